"""GPU: the probe read that allocates nothing (ms_sim_probe_read_static)
against the allocating ms_sim_probe_read, through the C ABI: identical
records on two calls in a row, the second smaller than the first (the shared
staging array keeps the first call's contents), and a clear error for a
record beyond the array."""
import ctypes as C

import numpy as np
import pytest

import paper_1805_11144_amd as M
from paper_1805_11144_amd import mergesim as MS
from synth import make_workload

pytestmark = pytest.mark.gpu


def _read_static(sim, probe, n_expected):
    out = np.full(n_expected, np.nan, np.float32)
    code = MS.load_library().ms_sim_probe_read_static(sim.handle, probe, out.ctypes.data_as(C.POINTER(C.c_float)),
                                                     out.size)
    return code, out


def test_static_read_equals_allocating_read_twice():
    w = make_workload("c2", n_steps=40, minibatch=3, n_neurons=20, n_eval=200)
    model = M.model_from_spec(w.spec)
    with M.Simulator(model, minibatch=w.minibatch, probe_capacity_steps=w.n_steps) as sim:
        sim.run_steps(w.n_steps, w.feeds)
        big = sim.data(0)                                     # allocating read
        code, got = _read_static(sim, 0, big.size)
        assert code == MS.MS_OK
        assert np.array_equal(got.reshape(big.shape), big)
        # a smaller record next: fewer steps after a reset
        sim.reset()
        k = 7
        sim.run_steps(k, {i: f[:, :k] for i, f in w.feeds.items()})
        small = sim.data(0)
        assert small.size < big.size
        code, got2 = _read_static(sim, 0, small.size)
        assert code == MS.MS_OK
        assert np.array_equal(got2.reshape(small.shape), small)
        # the binding's method returns the same
        assert np.array_equal(sim.data_static(0), small)


def test_static_read_rejects_records_beyond_the_array():
    """B * steps * width above PROBE_READ_STATIC_MAX is MS_E_INVALID with a
    message, and the allocating read still works."""
    w = make_workload("c2", n_steps=2, minibatch=64, n_neurons=10, n_eval=100)
    model = M.model_from_spec(w.spec)
    width = 64
    steps = MS.PROBE_READ_STATIC_MAX // (64 * width) + 1
    feeds = {i: np.repeat(f[:, :1], steps, axis=1) for i, f in w.feeds.items()}
    with M.Simulator(model, minibatch=64, probe_capacity_steps=steps) as sim:
        assert sim.probe_width(0) == width
        sim.run_steps(steps, feeds)
        n = 64 * steps * width
        assert n > MS.PROBE_READ_STATIC_MAX
        code, _ = _read_static(sim, 0, n)
        assert code == -1
        assert b"static staging array" in MS.load_library().ms_last_error()
        assert sim.data(0).shape == (64, steps, width)
