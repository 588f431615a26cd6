"""GPU: spike probes recorded as bitmasks (window driver, option
spike_probe_bits; paper Sec. 3.1: a spike probe records every neuron's output,
0 or amplitude / dt, at every step, so one bit per neuron and step holds it).

Checked through the C ABI against the float record of the same run without the
option (which the parity tests compare with the oracle):
  * the bit record read back as values (ms_sim_probe_read) equals the float
    record bit for bit;
  * its raw words (ms_sim_probe_read_bits) are the nonzero pattern of the float
    record, neuron 32 k + j in bit j of word k, the padding bits past the width 0;
  * probes of other targets keep their float records unchanged;
  * the same holds across runs split into several calls and through growth of
    the probe buffers (a small initial capacity);
  * drivers other than the window driver refuse the option, and a probe that is
    not bit-recorded refuses the bit read.
Shapes: the spiking classifier with 70-neuron layers (three words per step,
ragged), minibatch 8 and 5, and at the benchmark's size (784-1024-1024-10,
minibatch 256, 50 steps)."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from synth import make_workload

pytestmark = pytest.mark.gpu

MS = M.mergesim


def _run(w, bits, splits, cap):
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, driver=M.DRIVER_WINDOW,
                     probe_capacity_steps=cap, spike_probe_bits=bits) as sim:
        t0 = 0
        for n in splits:
            sim.run_steps(n, {i: f[:, t0:t0 + n] for i, f in w.feeds.items()})
            t0 += n
        data = [sim.data(p) for p in range(len(w.spec.probes))]
        words = {}
        if bits:
            for p in range(len(w.spec.probes)):
                try:
                    words[p] = sim.data_bits(p)
                except MS.MergesimError:
                    pass
    return data, words


def _unpack(words, width):
    j = np.arange(32, dtype=np.uint32)
    b = (words[..., None] >> j) & 1
    return b.reshape(words.shape[0], words.shape[1], -1)


def _compare(w, splits, cap):
    ref, _ = _run(w, False, splits, cap)
    got, words = _run(w, True, splits, cap)
    spike_probes = [p for p, pr in enumerate(w.spec.probes) if pr.target[0] == "neurons"]
    assert sorted(words) == spike_probes and len(spike_probes) >= 2
    for p in range(len(w.spec.probes)):
        np.testing.assert_array_equal(got[p], ref[p], err_msg=f"probe {p}")
    for p, wd in words.items():
        width = ref[p].shape[2]
        assert wd.shape == (w.minibatch, sum(splits), (width + 31) // 32)
        bitsv = _unpack(wd, width)
        np.testing.assert_array_equal(bitsv[..., :width], (ref[p] != 0).astype(np.uint32))
        assert not bitsv[..., width:].any()
        assert ref[p].any()   # the layer spiked: the comparison is not of zeros


@pytest.mark.parametrize("minibatch", [8, 5])
@pytest.mark.parametrize("splits,cap", [((37,), 1000), ((10, 27), 8)])
def test_bit_record_equals_float_record(minibatch, splits, cap):
    w = make_workload("c3", n_steps=sum(splits), minibatch=minibatch, n_in=40, n_hidden=70, n_out=6)
    _compare(w, splits, cap)


def test_bit_record_full_size():
    w = make_workload("c3")
    _compare(w, (w.n_steps,), 1000)


def test_refusals():
    w = make_workload("c3", n_steps=4, minibatch=2, n_in=8, n_hidden=40, n_out=3)
    with pytest.raises(MS.MergesimError):
        M.Simulator(M.model_from_spec(w.spec), minibatch=2, driver=M.DRIVER_GRAPH, spike_probe_bits=True)
    with M.Simulator(M.model_from_spec(w.spec), minibatch=2, driver=M.DRIVER_WINDOW) as sim:
        sim.run_steps(4, w.feeds)
        with pytest.raises(MS.MergesimError):
            sim.data_bits(0)
