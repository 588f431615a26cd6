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
