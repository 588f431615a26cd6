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
