"""Seeded random simulator state for injected-state tests (test input: shared
by the GPU run and the oracle; no simulation arithmetic)."""
import numpy as np


def random_state(spec, B, seed):
    """V in [0, 1), refractory time 0 for most neurons and U(0, tau_ref) for a
    quarter of them, filter states N(0, 0.3^2); keyed like OracleSim.get_state."""
    rng = np.random.default_rng(seed)
    st = {"V": {}, "ref": {}, "y": {}, "yp": {}}
    for i, e in enumerate(spec.ensembles):
        if e.neuron_type != "lif":
            continue
        st["V"][i] = rng.uniform(0.0, 1.0, (B, e.n_neurons)).astype(np.float32)
        ref = rng.uniform(0.0, e.tau_ref, (B, e.n_neurons))
        ref[rng.random((B, e.n_neurons)) < 0.75] = 0.0
        st["ref"][i] = ref.astype(np.float32)
    for ci, c in enumerate(spec.connections):
        if c.synapse is None:
            continue
        w = post_width(spec, c)
        st["y"][ci] = (0.3 * rng.standard_normal((B, w))).astype(np.float32)
    return st


def post_width(spec, c):
    """Width of the signal a connection writes into (its synapse state)."""
    if c.post_slice is not None:
        return c.post_slice[1] - c.post_slice[0]
    kind, i = c.post
    if kind == "node":
        return spec.nodes[i].size
    if kind == "ens":
        return spec.ensembles[i].dims
    return spec.ensembles[i].n_neurons
