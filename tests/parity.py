"""Parity metrics between the GPU simulator and the oracle (test helper)."""
import numpy as np


def rel_err(got, exp):
    """max |got - exp| / max |exp| (norm-relative, no division by zero)."""
    got = np.asarray(got, np.float64)
    exp = np.asarray(exp, np.float64)
    den = max(np.abs(exp).max(initial=0.0), 1e-30)
    return float(np.abs(got - exp).max(initial=0.0) / den)


def flip_fraction(got, exp):
    """Spike events present in exactly one of the two records, over the number
    of oracle spikes (a one-step shift counts twice)."""
    g = np.asarray(got) > 0
    e = np.asarray(exp) > 0
    return float(np.count_nonzero(g ^ e)) / max(1, int(np.count_nonzero(e)))


def unpaired_flips(got, exp):
    """Flipped spike events that are not one half of a one-step shift: a spike
    at step t in one record matched by a spike of the same neuron at t +- 1 in
    the other.  Rounding-level disagreement at the threshold only ever moves a
    spike by one step (the refractory period is measured from the interpolated
    crossing time), so every genuine flip is paired."""
    g = np.asarray(got) > 0
    e = np.asarray(exp) > 0
    only_g = g & ~e
    only_e = e & ~g
    def near(a, b):   # a-events with a b-event one step earlier or later
        m = np.zeros_like(a)
        m[:, 1:] |= b[:, :-1]
        m[:, :-1] |= b[:, 1:]
        return a & m
    return int(np.count_nonzero(only_g & ~near(only_g, only_e)) +
               np.count_nonzero(only_e & ~near(only_e, only_g)))


def lif_rate_inverse_ok(got, exp, J, scale, amp, tau_rc, tau_ref, rtol=1e-5):
    """Backward-error check of a rate-mode neuron probe.

    The rate r(J) has an unbounded slope at threshold (J -> 1+), and a neuron
    whose intercept is close to the radius has a very large gain, so float32
    rounding of J alone can move such a neuron's rate far beyond any forward
    tolerance.  An element passes if it is within rtol * max|exp| of the oracle
    (forward) or if it lies between amp*r(J - dJ) and amp*r(J + dJ) widened by
    rtol * max|exp|, with dJ = rtol * scale: the GPU value is then the exact
    rate of an input current that agrees with the oracle's to rtol relative to
    the size of the current's terms.  Returns (n_forward_fail, n_fail)."""
    from oracle.neurons import lif_rate
    got = np.asarray(got, np.float64)
    exp = np.asarray(exp, np.float64)
    tol = rtol * max(np.abs(exp).max(initial=0.0), 1e-30)
    fwd = np.abs(got - exp) <= tol
    dJ = rtol * scale
    lo = amp * lif_rate(J - dJ, tau_rc, tau_ref) - tol
    hi = amp * lif_rate(J + dJ, tau_rc, tau_ref) + tol
    ok = fwd | ((got >= lo) & (got <= hi))
    return int((~fwd).sum()), int((~ok).sum())


def lif_rate_spread(J, scale, amp, tau_rc, tau_ref, rtol=1e-5):
    """Largest change of amp*r(J) over currents within rtol*scale of J: the part
    of a rate neuron's output that float32 evaluation of its input current
    leaves undetermined (see lif_rate_inverse_ok)."""
    from oracle.neurons import lif_rate
    r0 = lif_rate(J, tau_rc, tau_ref)
    up = lif_rate(J + rtol * scale, tau_rc, tau_ref) - r0
    dn = r0 - lif_rate(J - rtol * scale, tau_rc, tau_ref)
    return amp * np.maximum(up, dn)
