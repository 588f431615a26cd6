"""GPU: the fused synapse filter + scatter-accumulate launch (MS_FUSE_SYNAPSES)
against the same simulation with the connections' DotInc, Lowpass, Reset and
CopyInc as separate launches.  The fused kernel sums in the same order as the
separate ones (transform in k order, filter update, copy in CopyInc order), so
the probes must agree bit for bit, and both must match the oracle at the
rate-mode bound (the oracle comparison of every driver is in
test_gpu_parity.py)."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from oracle.sim import OracleSim
from synth import make_workload
from tests.parity import rel_err

pytestmark = pytest.mark.gpu

BOTH = M.mergesim.FUSE_ENSEMBLES | M.mergesim.FUSE_SYNAPSES
ENS_ONLY = M.mergesim.FUSE_ENSEMBLES
SMALL = {
    "c1": dict(n_steps=200),
    "c4": dict(n_steps=60, minibatch=3, n_ens=6, n_neurons=40, n_eval=200),
    "c5": dict(n_steps=40, n_ens=12, n_neurons=40, n_eval=200, n_input_targets=4, n_probed=3),
}
DRIVERS = {"steps": M.DRIVER_STEPS, "graph": M.DRIVER_GRAPH}


def _run(w, fuse, driver, split=None):
    model = M.model_from_spec(w.spec)
    with M.Simulator(model, minibatch=w.minibatch, driver=driver, unroll=7, fuse=fuse,
                     probe_capacity_steps=w.n_steps) as sim:
        info = sim.info()
        if split is None:
            sim.run_steps(w.n_steps, w.feeds)
        else:
            sim.run_steps(split, {i: f[:, :split] for i, f in w.feeds.items()})
            sim.run_steps(w.n_steps - split, {i: f[:, split:] for i, f in w.feeds.items()})
        return [sim.data(p) for p in range(len(w.spec.probes))], info


@pytest.mark.parametrize("neuron_type", ["lif", "lif_rate"])
@pytest.mark.parametrize("driver", list(DRIVERS))
@pytest.mark.parametrize("name", list(SMALL))
def test_fused_equals_separate(name, driver, neuron_type):
    w = make_workload(name, neuron_type=neuron_type, **SMALL[name])
    got, gi = _run(w, BOTH, DRIVERS[driver], split=w.n_steps // 3)
    exp, ei = _run(w, ENS_ONLY, DRIVERS[driver])
    print(f"{name} {driver} {neuron_type}: groups per step {ei['groups_per_step']} -> {gi['groups_per_step']}")
    assert gi["groups_per_step"] < ei["groups_per_step"]
    for pi, (g, e) in enumerate(zip(got, exp)):
        d = float(np.abs(g.astype(np.float64) - e).max())
        print(f"  probe {pi}: max |fused - separate| = {d:.3e}")
        assert np.array_equal(g, e), (name, driver, neuron_type, pi, d)


def test_fused_full_size_sparse_graph():
    """The full 5000-ensemble graph for 60 steps in the benchmark's launch
    configuration (hipGraph, 20 steps per launch): fused equals separate bit
    for bit, and the step runs 2 launches."""
    w = make_workload("c5", n_steps=60)
    model = M.model_from_spec(w.spec)
    outs = []
    for fuse in (BOTH, ENS_ONLY):
        with M.Simulator(model, driver=M.DRIVER_GRAPH, unroll=20, fuse=fuse, probe_capacity_steps=60) as sim:
            sim.run_steps(w.n_steps, w.feeds)
            outs.append(([sim.data(p) for p in range(len(w.spec.probes))], sim.info()))
    (got, gi), (exp, ei) = outs
    print(f"groups per step {ei['groups_per_step']} -> {gi['groups_per_step']}")
    assert gi["groups_per_step"] == 2   # ensembles, fused synapses (the feed and probe fold in)
    for pi, (g, e) in enumerate(zip(got, exp)):
        assert np.array_equal(g, e), pi


@pytest.mark.parametrize("driver", list(DRIVERS))
def test_injected_synapse_state_is_pulled(driver):
    """A synapse state written between runs (ms_sim_set_state) reaches the post
    input of the next step: the run's first launch pulls the post inputs from
    the filter state.  Checked against the oracle given the same state."""
    w = make_workload("c5", neuron_type="lif_rate", **SMALL["c5"])
    model = M.model_from_spec(w.spec)
    rng = np.random.default_rng(7)
    conns = [i for i, c in enumerate(w.spec.connections) if c.synapse is not None]
    ref = OracleSim(w.spec, minibatch=w.minibatch, param_dtype=np.float32)
    with M.Simulator(model, minibatch=w.minibatch, driver=DRIVERS[driver], unroll=7, fuse=BOTH,
                     probe_capacity_steps=w.n_steps) as sim:
        k = 10
        sim.run_steps(k, {i: f[:, :k] for i, f in w.feeds.items()})
        ref.run_steps(k, {i: f[:, :k] for i, f in w.feeds.items()})
        for c in conns[:5]:
            width = ref.y[c].shape[1]
            val = rng.uniform(-1, 1, size=(w.minibatch, width)).astype(np.float32)
            sim.set_state(M.mergesim.STATE_SYNAPSE, c, val)
            ref.y[c][...] = val
        sim.run_steps(w.n_steps - k, {i: f[:, k:] for i, f in w.feeds.items()})
        ref.run_steps(w.n_steps - k, {i: f[:, k:] for i, f in w.feeds.items()})
        for p in range(len(w.spec.probes)):
            r = rel_err(sim.data(p), ref.data(p))
            print(f"probe {p}: rel {r:.2e}")
            assert r <= 1e-5, (p, r)
