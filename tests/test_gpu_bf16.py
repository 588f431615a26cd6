"""bf16 window products against the oracle.

The paper lets the user pick the simulation dtype (Sec. 3.1: float32 or
float64); bf16 inputs with fp32 accumulation are this library's addition for
the matrix cores.  With gemm_dtype="bf16" the simulator rounds the weights of
its large products (M >= 64, K >= 16, K % 8 == 0, minibatch % 4 == 0) to bf16
once, and their signal operand as it is read.

In the spiking classifier every such signal operand is exact in bf16: the
input images are rounded to bf16 here before either side sees them, and the
hidden layers' spikes are 0 or amplitude/dt = 1000 (seven significant bits).
So the oracle, handed the same bf16-rounded weights, computes the same products
up to fp32 summation order, and the fp32 spiking bounds apply unchanged.  The
rounding below is the input transformation both sides are fed; it is not part
of either implementation."""
import copy

import numpy as np
import pytest

import paper_1805_11144_amd as M
from oracle.sim import OracleSim
from synth import make_workload
from tests.parity import check_spiking_probe, flip_fraction, float32_run
from tests.test_gpu_shadow import compare_step, full_state, oracle_step

pytestmark = pytest.mark.gpu


def round_bf16(a):
    """float32 values rounded to the nearest bf16 (ties to even), as float64."""
    u = np.asarray(a, np.float32).view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def bf16_inputs(w):
    """The workload with bf16-exact feeds, and the spec the oracle sees: the
    transforms of the products that run on bf16 rounded."""
    w = copy.deepcopy(w)
    w.feeds = {k: round_bf16(v).astype(np.float32) for k, v in w.feeds.items()}
    ospec = copy.deepcopy(w.spec)
    rounded = []
    for ci, c in enumerate(ospec.connections):
        t = np.asarray(c.transform)
        if t.ndim == 2 and t.shape[0] >= 64 and t.shape[1] >= 16 and t.shape[1] % 8 == 0 \
                and w.minibatch % 4 == 0:
            c.transform = round_bf16(t)
            rounded.append(ci)
    return w, ospec, rounded


def gpu_run(w, **opts):
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, unroll=20,
                     probe_capacity_steps=w.n_steps, **opts) as sim:
        sim.run_steps(w.n_steps, w.feeds)
        return [sim.data(p) for p in range(len(w.spec.probes))]


def oracle_run(spec, w):
    ref = OracleSim(spec, minibatch=w.minibatch, param_dtype=np.float32)
    ref.run_steps(w.n_steps, w.feeds)
    return [ref.data(p) for p in range(len(spec.probes))]


# several 128 x 128 tiles with ragged edges in M (200), K (136 = 4 slices of 32
# + 8) and the window's columns (20 steps x 12)
SMALL = dict(n_steps=20, minibatch=12, n_hidden=200, n_in=136)


def test_bf16_spiking_matches_oracle_with_rounded_weights():
    w, ospec, rounded = bf16_inputs(make_workload("c3", neuron_type="lif", **SMALL))
    assert rounded == [0, 1]                 # W1 and W2; the 10-row readout stays fp32
    got = gpu_run(w, gemm_dtype="bf16")
    exp = oracle_run(ospec, w)
    exp_f32 = oracle_run(w.spec, w)
    floor = float32_run(ospec, w.minibatch, w.n_steps, w.feeds)
    control = 0
    for pi, (g, e, e32, fl) in enumerate(zip(got, exp, exp_f32, floor)):
        p = w.spec.probes[pi]
        check_spiking_probe(f"probe {pi}", p, g, e, fl)
        if p.target[0] == "neurons":
            print(f"  against unrounded weights: flips {flip_fraction(g, e32):.2e}")
            control += flip_fraction(g, e32) > 2e-3
    # control: the products really ran in bf16 -- against the oracle with the
    # unrounded weights far more spikes disagree
    assert control >= 1


def test_ineligible_products_stay_fp32():
    """minibatch 6 is not a multiple of 4: every product keeps fp32, so the
    results match the oracle with the original weights."""
    w = make_workload("c3", neuron_type="lif", **{**SMALL, "minibatch": 6})
    w, ospec, rounded = bf16_inputs(w)
    assert rounded == []
    got = gpu_run(w, gemm_dtype="bf16")
    exp = oracle_run(w.spec, w)
    floor = float32_run(w.spec, w.minibatch, w.n_steps, w.feeds)
    for pi, (g, e, fl) in enumerate(zip(got, exp, floor)):
        check_spiking_probe(f"probe {pi}", w.spec.probes[pi], g, e, fl)


def test_bf16_needs_the_window_driver():
    w = make_workload("c3", neuron_type="lif", **SMALL)
    with pytest.raises(M.MergesimError, match="window driver"):
        M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, driver=M.DRIVER_STEPS,
                    gemm_dtype="bf16")
    with pytest.raises(M.MergesimError, match="gemm_dtype"):
        M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, gemm_dtype=7)


@pytest.mark.timeout(900)
def test_bf16_full_size_one_step():
    """The full classifier (784-1024-1024-10, minibatch 256) in the benchmark's
    launch configuration: one oracle step from the GPU's state at sampled steps,
    with the spiking bounds of the fp32 path."""
    w, ospec, rounded = bf16_inputs(make_workload("c3", neuron_type="lif"))
    assert rounded == [0, 1]
    ref = OracleSim(ospec, minibatch=w.minibatch, param_dtype=np.float32,
                    record_current=tuple(range(len(ospec.ensembles))))
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, unroll=20,
                     probe_capacity_steps=w.n_steps, gemm_dtype="bf16") as sim:
        cur = 0
        for k in [0, 1, 10, 49]:
            if k > cur:
                sim.run_steps(k - cur, {n: f[:, cur:k] for n, f in w.feeds.items()})
            st0 = full_state(sim, w.spec, w.minibatch, True)
            sim.run_steps(1, {n: f[:, k:k + 1] for n, f in w.feeds.items()})
            cur = k + 1
            st1 = full_state(sim, w.spec, w.minibatch, True)
            probes1 = [sim.data(p)[:, k] for p in range(len(w.spec.probes))]
            oracle_step(ref, w, st0, k)
            s = compare_step(w, st0, st1, probes1, ref, True)
            print(f"bf16 k={k}: disagree {s['disagree']} of {s['spikes']} spikes, "
                  f"y err {s['y_err']:.2e}, probe err {s['probe_err']:.2e}", flush=True)
            assert s["disagree"] <= max(2, 1e-4 * s["spikes"])
            assert s["y_err"] <= 1e-3 and s["probe_err"] <= 1e-3
