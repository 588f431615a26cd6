"""GPU: PES online learning (paper Sec. 5.1, the pes benchmark; Fig. 7: one
weight matrix per batch element) against the oracle, through the C ABI.

Compared: every probe, and the learned decoders themselves after the run
(ms_sim_get_state MS_STATE_LEARNED_DECODERS), element by element.  Bounds as
for every other model: rate mode within 1e-5 of the peak or twice the
float32-arithmetic oracle's deviation (the decoders integrate float32
rounding of every error and activity product over the run); spiking runs
within the stated spike/filtered bounds or twice the float32 floor
(tests/parity.py).  Both GPU paths are covered: the decode and the update in
one pass over the decoders (filtered error connections: the error is known
when the decode runs) and as two launches (unfiltered error path)."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from oracle.sim import OracleSim
from synth import make_workload
from tests.parity import FLOOR_FACTOR, RATE_REL, check_rate_probe, check_spiking_probe, rel_err
from tests.test_pes_plan import _learned_solved

pytestmark = pytest.mark.gpu

MS = M.mergesim
SMALL = dict(n_steps=200, minibatch=3, D=8, neurons_per_dim=80, learning_rate=5e-4)   # 640 neurons
DRIVERS = {"steps": M.DRIVER_STEPS, "graph": M.DRIVER_GRAPH}


def _gpu(spec, B, T, feeds, split=None, **opts):
    with M.Simulator(M.model_from_spec(spec), minibatch=B, probe_capacity_steps=T, unroll=7, **opts) as sim:
        if split is None:
            sim.run_steps(T, feeds)
        else:
            sim.run_steps(split, {i: f[:, :split] for i, f in feeds.items()})
            sim.run_steps(T - split, {i: f[:, split:T] for i, f in feeds.items()})
        out = [sim.data(p) for p in range(len(spec.probes))]
        W = {c: sim.get_state(MS.STATE_LEARNED_DECODERS, c,
                              spec.ensembles[spec.connections[c].pre[1]].n_neurons * _k(spec, c))
             for c, cc in enumerate(spec.connections) if cc.learning_rule is not None}
        info = sim.info()
    return out, W, info


def _k(spec, c):
    cc = spec.connections[c]
    if cc.decoders is not None:
        return np.asarray(cc.decoders).shape[1]
    return spec.ensembles[cc.pre[1]].dims


def _oracle(spec, B, T, feeds, arith=np.float64):
    ref = OracleSim(spec, minibatch=B, param_dtype=np.float32, arith_dtype=arith)
    ref.run_steps(T, {i: f[:, :T] for i, f in feeds.items()})
    return [ref.data(p) for p in range(len(spec.probes))], {c: W.reshape(B, -1) for c, W in ref.W.items()}


def _check_all(tag, spec, got, Wg, exp, We, f32, Wf, spiking):
    for pi, (g, e, f) in enumerate(zip(got, exp, f32)):
        if spiking:
            check_spiking_probe(f"{tag} probe {pi}", spec.probes[pi], g, e, f)
        else:
            check_rate_probe(f"{tag} probe {pi}", g, e, f)
    for c in We:
        r, floor = rel_err(Wg[c], We[c]), rel_err(Wf[c], We[c])
        bound = max(RATE_REL, FLOOR_FACTOR * floor) if not spiking else max(1e-3, FLOOR_FACTOR * floor)
        print(f"{tag} decoders of connection {c}: rel {r:.2e} (float32 floor {floor:.2e}, bound {bound:.2e})")
        assert r <= bound, (tag, c, r, bound)


@pytest.mark.parametrize("neuron_type", ["lif_rate", "lif"])
@pytest.mark.parametrize("driver", list(DRIVERS))
def test_pes_workload_parity(driver, neuron_type):
    w = make_workload("pes", neuron_type=neuron_type, **SMALL)
    got, Wg, info = _gpu(w.spec, w.minibatch, w.n_steps, w.feeds, split=w.n_steps // 3, driver=DRIVERS[driver])
    exp, We = _oracle(w.spec, w.minibatch, w.n_steps, w.feeds)
    f32, Wf = _oracle(w.spec, w.minibatch, w.n_steps, w.feeds, np.float32)
    print(f"pes {driver} {neuron_type}: {info['groups_per_step']} launches per step")
    _check_all(f"pes {driver} {neuron_type}", w.spec, got, Wg, exp, We, f32, Wf, neuron_type == "lif")
    # the decoders learned (they started at zero) and differ between batch rows
    W = Wg[1]
    assert np.abs(W).max() > 0 and np.abs(W[0] - W[1]).max() > 1e-3 * np.abs(W).max()


@pytest.mark.parametrize("pre_synapse", [0.005, None])
@pytest.mark.parametrize("err_synapse", [0.005, None])
def test_solved_decoders_fused_and_separate_update(err_synapse, pre_synapse):
    """Filtered error: decode and update in one pass; unfiltered: two launches."""
    spec, feeds, B, T = _learned_solved("lif_rate", pre_synapse, err_synapse, None if err_synapse is None else 0.005)
    got, Wg, _ = _gpu(spec, B, T, feeds, driver=M.DRIVER_STEPS)
    exp, We = _oracle(spec, B, T, feeds)
    f32, Wf = _oracle(spec, B, T, feeds, np.float32)
    _check_all(f"solved err={err_synapse} pre={pre_synapse}", spec, got, Wg, exp, We, f32, Wf, False)


def test_reset_restores_and_state_round_trips():
    w = make_workload("pes", neuron_type="lif_rate", **SMALL)
    n = w.spec.ensembles[0].n_neurons * 8
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, probe_capacity_steps=w.n_steps) as sim:
        W0 = sim.get_state(MS.STATE_LEARNED_DECODERS, 1, n)
        assert not W0.any()                                   # zero initial decoders
        sim.run_steps(50, {i: f[:, :50] for i, f in w.feeds.items()})
        W1 = sim.get_state(MS.STATE_LEARNED_DECODERS, 1, n)
        A1 = sim.get_state(MS.STATE_PES_ACTIVITY, 1, w.spec.ensembles[0].n_neurons)
        assert np.abs(W1).max() > 0 and np.abs(A1).max() > 0
        rng = np.random.default_rng(1)
        inj = rng.normal(0, 1e-4, W1.shape).astype(np.float32)
        sim.set_state(MS.STATE_LEARNED_DECODERS, 1, inj)
        np.testing.assert_array_equal(sim.get_state(MS.STATE_LEARNED_DECODERS, 1, n), inj)
        sim.reset()
        assert not sim.get_state(MS.STATE_LEARNED_DECODERS, 1, n).any()
        sim.run_steps(50, {i: f[:, :50] for i, f in w.feeds.items()})
        np.testing.assert_array_equal(sim.get_state(MS.STATE_LEARNED_DECODERS, 1, n), W1)


def test_injected_decoders_parity():
    """Decoders injected between runs (ms_sim_set_state) are the ones the next
    run decodes with and updates, as in the oracle given the same values."""
    w = make_workload("pes", neuron_type="lif_rate", **SMALL)
    B, D = w.minibatch, 8
    n = w.spec.ensembles[0].n_neurons
    rng = np.random.default_rng(5)
    inj = rng.normal(0, 2e-4, (B, n * D)).astype(np.float32)
    ref = OracleSim(w.spec, minibatch=B, param_dtype=np.float32)
    ref32 = OracleSim(w.spec, minibatch=B, arith_dtype=np.float32)
    with M.Simulator(M.model_from_spec(w.spec), minibatch=B, probe_capacity_steps=w.n_steps) as sim:
        k = 20
        sim.run_steps(k, {i: f[:, :k] for i, f in w.feeds.items()})
        for r in (ref, ref32):
            r.run_steps(k, {i: f[:, :k] for i, f in w.feeds.items()})
            r.W[1] = inj.reshape(B, n, D).astype(r.dtype)
        sim.set_state(MS.STATE_LEARNED_DECODERS, 1, inj)
        rest = {i: f[:, k:] for i, f in w.feeds.items()}
        sim.run_steps(w.n_steps - k, rest)
        for r in (ref, ref32):
            r.run_steps(w.n_steps - k, rest)
        got = sim.data(0)
    check_rate_probe("pes injected decoders", got, ref.data(0), ref32.data(0))


@pytest.mark.parametrize("driver", [M.DRIVER_PERSISTENT, M.DRIVER_WINDOW])
def test_other_drivers_refuse_learning(driver):
    w = make_workload("pes", **SMALL)
    with pytest.raises(MS.MergesimError):
        M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, driver=driver)


@pytest.mark.timeout(900)
def test_pes_full_size_sampled_rows():
    """The benchmark workload (D = 192, 9600 neurons, 10 batch rows, 1000
    steps) in the benchmark's launch configuration; the oracle on 2 of the
    10 rows (rows are independent: each learns its own decoders)."""
    w = make_workload("pes")
    rows = np.array([0, 7])
    got, Wg, info = _gpu(w.spec, w.minibatch, w.n_steps, w.feeds)
    assert info["driver"] == M.DRIVER_GRAPH
    feeds = {i: f[rows] for i, f in w.feeds.items()}
    exp, We = _oracle(w.spec, len(rows), w.n_steps, feeds)
    f32, Wf = _oracle(w.spec, len(rows), w.n_steps, feeds, np.float32)
    _check_all("pes full", w.spec, [g[rows] for g in got], {c: W[rows] for c, W in Wg.items()},
               exp, We, f32, Wf, True)
