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


# ------------------------------------------------------------- whole-run bounds
# Over a whole run, float32 arithmetic by itself moves spikes across the
# threshold (the state drifts from its float64 value step by step), and a
# moved spike shifts every filtered value downstream by (1 - a) amplitude/dt
# times a decoder weight.  The oracle run in float32 arithmetic (OracleSim with
# arith_dtype=float32, the plainest float32 simulator) measures that floor on
# the same inputs.  A whole-run comparison holds the GPU to the stated bound or
# to FLOOR_FACTOR times the float32 floor, whichever is larger.
FLOOR_FACTOR = 2.0
SPIKE_FLIPS = 1e-4      # spike events flipped, of the oracle's spikes
FILTERED_ABS = 1e-3     # filtered / decoded probe outputs, absolute
RATE_REL = 1e-5         # rate-mode probes, relative to the probe's peak


def float32_run(spec, B, n_steps, feeds, state=None):
    """Probe records of the oracle run in float32 arithmetic (from `state`,
    keyed like OracleSim.get_state, if given)."""
    from oracle.sim import OracleSim
    ref = OracleSim(spec, minibatch=B, arith_dtype=np.float32)
    if state is not None:
        ref.set_state(state)
    ref.run_steps(n_steps, {k: f[:, :n_steps] for k, f in feeds.items()})
    return [ref.data(p) for p in range(len(spec.probes))]


def check_spiking_probe(tag, probe, got, exp, f32):
    """Spiking-mode bound of one probe record: spike flips against the oracle
    within max(SPIKE_FLIPS, FLOOR_FACTOR x the float32 run's flips); any other
    probe (decoded, node, filtered) within max(FILTERED_ABS, FLOOR_FACTOR x the
    float32 run's largest deviation)."""
    if probe.target[0] == "neurons":
        f, floor = flip_fraction(got, exp), flip_fraction(f32, exp)
        bound = max(SPIKE_FLIPS, FLOOR_FACTOR * floor)
        print(f"{tag}: flips {f:.2e} of {int((np.asarray(exp) > 0).sum())} spikes (float32 floor {floor:.2e}, "
              f"bound {bound:.2e}), unpaired {unpaired_flips(got, exp)}")
        assert f <= bound, (tag, f, bound)
    else:
        d = float(np.abs(np.asarray(got, np.float64) - exp).max(initial=0.0))
        floor = float(np.abs(np.asarray(f32, np.float64) - exp).max(initial=0.0))
        bound = max(FILTERED_ABS, FLOOR_FACTOR * floor)
        print(f"{tag}: abs {d:.2e} (float32 floor {floor:.2e}, bound {bound:.2e})")
        assert d <= bound, (tag, d, bound)


def check_rate_probe(tag, got, exp, f32):
    """Rate-mode bound of a decoded or node probe: relative error within
    max(RATE_REL, FLOOR_FACTOR x the float32 run's relative error)."""
    r, floor = rel_err(got, exp), rel_err(f32, exp)
    bound = max(RATE_REL, FLOOR_FACTOR * floor)
    print(f"{tag}: rel {r:.2e} (float32 floor {floor:.2e}, bound {bound:.2e})")
    assert r <= bound, (tag, r, bound)


# ------------------------------------------------- the first spike disagreement
EPS32 = 2.0 ** -24


def first_flip(gpu_spikes, exp_spikes):
    """(ensemble, step, batch row, neuron) of the earliest spike on which two
    records of every ensemble's spikes ({ensemble: [B, T, n]}) disagree, or
    None."""
    first = None
    for e, g in gpu_spikes.items():
        d = np.argwhere((np.asarray(g) > 0) != (np.asarray(exp_spikes[e]) > 0))
        if len(d):
            b, t, n = d[np.argmin(d[:, 1])]
            if first is None or t < first[1]:
                first = (e, int(t), int(b), int(n))
    return first


def flip_explained(V, ref, J, scale, dt, tau_rc):
    """Whether a spike decision lies within float32 resolution of the
    threshold: the voltage before the threshold test, computed in float64 from
    the oracle's state (V, refractory time) and current J, is within the band
    a float32 evaluation can move it -- the current's rounding, 8 eps32 times
    the size of its terms (scale: |bias| + |x| |E| + |gain| |input|), through
    the integration factor, plus 16 eps32 of the voltage's own rounding.
    Returns (explained, margin, band)."""
    integ = min(max(dt - ref, 0.0), dt)
    e = -np.expm1(-integ / tau_rc)
    pre = V + (J - V) * e
    band = e * 8 * EPS32 * scale + 16 * EPS32
    return abs(pre - 1.0) <= band, pre - 1.0, band
