"""CPU tests of the stage-major (window) schedule: which models qualify, and
that running the exported schedule -- every phase over a whole window of
steps, versioned signals, private neuron state -- in float64 equals the
unmerged oracle step by step."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from oracle.sim import OracleSim
from synth import make_workload
from tests.plan_exec import WindowExecutor
from tests.test_plan_cpu import SMALL


def window_of(name, **opts):
    w = make_workload(name, **SMALL[name])
    return w, M.Plan(M.model_from_spec(w.spec), minibatch=w.minibatch, **opts).json()["window"]


@pytest.mark.parametrize("name", ["c1", "c5", "bg"])
def test_recurrent_models_are_refused(name):
    _, win = window_of(name)
    assert not win["ok"] and "cycle" in win["why"]


@pytest.mark.parametrize("name", ["c2", "c3", "c4"])
def test_schedule_covers_every_operator_once_in_level_order(name):
    w, win = window_of(name)
    plan = M.Plan(M.model_from_spec(w.spec), minibatch=w.minibatch).json()
    all_ops = sorted(o for g in plan["groups"] for o in g["ops"])
    ph_ops = sorted(o for ph in win["phases"] for o in ph["group"]["ops"])
    assert ph_ops == all_ops
    levels = [ph["level"] for ph in win["phases"]]
    assert levels == sorted(levels)
    # neuron state is private, everything a probe reads is versioned
    assert win["rows_p"] == 2 * sum(e.n_neurons for e in w.spec.ensembles if e.neuron_type == "lif")


def test_chain_levels_follow_the_chain():
    """In the ensemble chain every link adds levels: ensemble i+1 runs after i."""
    w, win = window_of("c4")
    first = {}
    for ph in win["phases"]:
        for o in ph["group"]["ops"]:
            if o.endswith(".ens"):
                first[int(o.split(".")[0][1:])] = ph["level"]
    lv = [first[i] for i in sorted(first)]
    assert all(b > a for a, b in zip(lv, lv[1:]))


@pytest.mark.parametrize("name", ["c2", "c3", "c4"])
@pytest.mark.parametrize("neuron_type", ["lif_rate", "lif", "relu"])
@pytest.mark.parametrize("window", [1, 7, 1000])
@pytest.mark.parametrize("opts", [dict(), dict(fuse=False), dict(merge=False)])
def test_window_execution_matches_oracle(name, neuron_type, window, opts):
    w = make_workload(name, neuron_type=neuron_type, **SMALL[name])
    plan = M.Plan(M.model_from_spec(w.spec), minibatch=w.minibatch, **opts)
    ref = OracleSim(w.spec, minibatch=w.minibatch, param_dtype=np.float32)
    ex = WindowExecutor(plan, w.spec, w.minibatch, window, params_from=ref)
    ex.run(w.n_steps, w.feeds)
    ref.run_steps(w.n_steps, w.feeds)
    for pi in range(len(w.spec.probes)):
        got, exp = ex.data(pi), ref.data(pi)
        assert got.shape == exp.shape
        scale = max(1.0, np.abs(exp).max())
        if neuron_type == "lif" and w.spec.probes[pi].target[0] == "neurons":
            assert np.array_equal(got > 0, exp > 0)
        np.testing.assert_allclose(got, exp, rtol=0, atol=1e-11 * scale)


CHAIN = dict(n_steps=60, minibatch=2, n_ens=4, n_neurons=150, n_eval=200)


@pytest.mark.parametrize("neuron_type", ["lif_rate", "lif", "relu"])
@pytest.mark.parametrize("window", [1, 7, 1000])
def test_connection_chains_fuse_into_the_ensembles(neuron_type, window):
    """Wide-array links (transform DotInc -> lowpass -> copy into the next
    ensemble's only input, Fig. 2) fuse into the next ensemble's window phase:
    their three phases and the resets of v and x leave the schedule, the
    ensemble computes x_t = y_{t-1}, y_t = a y_{t-1} + b W d_t itself, and the
    run still equals the unmerged oracle."""
    w = make_workload("c4", neuron_type=neuron_type, **CHAIN)
    plan = M.Plan(M.model_from_spec(w.spec), minibatch=w.minibatch)
    win = plan.json()["window"]
    chained = [ph["group"]["ops"][0] for ph in win["phases"] if "chain" in ph["group"]]
    assert chained == ["e1.ens", "e2.ens", "e3.ens"]
    ops = {o for ph in win["phases"] for o in ph["group"]["ops"]}
    for c in (1, 2, 3):   # the links into e1..e3 are connections 1..3
        assert not {f"c{c}.transform", f"c{c}.synapse", f"c{c}.deliver", f"c{c}.resetv"} & ops
        assert f"e{c}.resetx" not in ops
    ref = OracleSim(w.spec, minibatch=w.minibatch, param_dtype=np.float32)
    ex = WindowExecutor(plan, w.spec, w.minibatch, window, params_from=ref)
    half = w.n_steps // 2
    ex.run(half, {i: f[:, :half] for i, f in w.feeds.items()})
    ex.run(w.n_steps - half, {i: f[:, half:] for i, f in w.feeds.items()})
    ref.run_steps(w.n_steps, w.feeds)
    for pi in range(len(w.spec.probes)):
        got, exp = ex.data(pi), ref.data(pi)
        scale = max(1.0, np.abs(exp).max())
        np.testing.assert_allclose(got, exp, rtol=0, atol=1e-11 * scale)


def test_chains_need_one_column_per_workgroup():
    """Ensembles of at most 128 neurons share a workgroup between batch
    columns (minibatch > 1), and ensembles of more than 512 take several
    neurons per thread: no fusion there."""
    w = make_workload("c4", **{**CHAIN, "n_neurons": 100})
    win = M.Plan(M.model_from_spec(w.spec), minibatch=w.minibatch).json()["window"]
    assert not any("chain" in ph["group"] for ph in win["phases"])
    w1 = make_workload("c4", **{**CHAIN, "n_neurons": 100, "minibatch": 1})
    win1 = M.Plan(M.model_from_spec(w1.spec), minibatch=1).json()["window"]
    assert sum("chain" in ph["group"] for ph in win1["phases"]) == 3
    for n, fused in ((512, 3), (513, 0)):
        wn = make_workload("c4", **{**CHAIN, "n_neurons": n, "n_eval": 50})
        winn = M.Plan(M.model_from_spec(wn.spec), minibatch=wn.minibatch).json()["window"]
        assert sum("chain" in ph["group"] for ph in winn["phases"]) == fused, n
