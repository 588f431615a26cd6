"""The library's C++ planner against the independent reference planner: the
exported plans (signal layout, merged groups, operator order, index arrays)
must be identical."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from oracle import planner_ref as P
from synth import make_workload

CASES = {
    "c1": dict(),
    "c2": dict(n_steps=2, minibatch=1, n_neurons=20, n_eval=50),
    "c3": dict(n_steps=2, minibatch=1, n_hidden=64, n_in=30),
    "c4": dict(n_steps=2, minibatch=1, n_ens=12, n_neurons=30, n_eval=40),
    "c5": dict(n_steps=2, n_ens=15, n_neurons=30, n_eval=40, n_input_targets=5, n_probed=4),
    "bg": dict(n_steps=2, D=5, n_neurons=20, n_eval=40),
    "pes": dict(n_steps=2, minibatch=2, D=6, neurons_per_dim=5),
}
FLOAT_KEYS = {"values", "tau_rc", "tau_ref", "amp", "ca", "cb", "coef", "sigma"}


def _strip(plan):
    plan = dict(plan)
    plan.pop("window", None)   # the stage-major schedule is checked in test_window_plan.py
    plan.pop("launch", None)   # the time-major step program is checked in test_launch_plan.py
    plan["groups"] = [{k: v for k, v in g.items() if k not in FLOAT_KEYS} for g in plan["groups"]]
    return plan


OPTS = {
    "tree3": (dict(), dict()),
    "greedy": (dict(planner=M.PLANNER_GREEDY), dict(planner="greedy")),
    "tree2_nosort": (dict(planner_depth=2, sort=False), dict(depth=2, sort=False)),
    "nosimplify": (dict(simplify=False), dict(do_simplify=False)),
    "nomerge": (dict(merge=False), dict(merge=False)),
    "nofuse": (dict(fuse=False), dict(fuse=False)),
}


@pytest.mark.parametrize("name", ["c1", "c2", "c3", "c4"])
def test_full_size_plans_identical(name):
    """Full benchmark-size models (default options)."""
    w = make_workload(name)
    got = _strip(M.Plan(M.model_from_spec(w.spec)).json())
    exp = P.make_plan(w.spec)
    assert got == {**exp, "groups": exp["groups"]}


@pytest.mark.parametrize("opt", list(OPTS))
@pytest.mark.parametrize("name", list(CASES))
def test_plans_identical(name, opt):
    w = make_workload(name, **CASES[name])
    lib_opts, ref_opts = OPTS[opt]
    got = _strip(M.Plan(M.model_from_spec(w.spec), **lib_opts).json())
    exp = P.make_plan(w.spec, **ref_opts)
    assert got["bases"] == exp["bases"]
    assert got["signals"] == exp["signals"]
    assert len(got["groups"]) == len(exp["groups"])
    for g, e in zip(got["groups"], exp["groups"]):
        assert g == e
    assert got["probe_rows"] == exp["probe_rows"]
    assert got["probe_offsets"] == exp["probe_offsets"]
    assert got["feed_rows"] == exp["feed_rows"]


@pytest.mark.parametrize("opt", ["tree3", "nofuse", "nomerge"])
@pytest.mark.parametrize("name", ["c2", "c4", "c5"])
def test_relu_plans_identical(name, opt):
    """ReLU ensembles: rate operators keyed and exported with their neuron type."""
    w = make_workload(name, neuron_type="relu", **CASES[name])
    lib_opts, ref_opts = OPTS[opt]
    got = _strip(M.Plan(M.model_from_spec(w.spec), **lib_opts).json())
    exp = P.make_plan(w.spec, **ref_opts)
    assert got == {**exp, "groups": exp["groups"]}
    kinds = [g.get("neuron") for g in got["groups"] if g["type"] in ("SimLIFRate", "Ensemble")]
    assert kinds and all(k == 2 for k in kinds)


@pytest.mark.parametrize("opt", ["tree3", "nofuse", "nomerge"])
@pytest.mark.parametrize("name", ["c2", "c4", "c5"])
def test_soft_lif_rate_plans_identical(name, opt):
    """Soft LIF rate ensembles: never fused, their rate operators keyed and
    exported with the neuron type (the smoothing travels per row)."""
    w = make_workload(name, neuron_type="softlif_rate", **CASES[name])
    lib_opts, ref_opts = OPTS[opt]
    full = M.Plan(M.model_from_spec(w.spec), **lib_opts).json()
    got = _strip(full)
    exp = P.make_plan(w.spec, **ref_opts)
    assert got == {**exp, "groups": exp["groups"]}
    assert not [g for g in got["groups"] if g["type"] == "Ensemble"]
    rate = [g for g in full["groups"] if g["type"] == "SimLIFRate"]
    assert rate and all(g["neuron"] == 3 for g in rate)
    assert all(np.allclose(g["sigma"], w.spec.ensembles[0].sigma) for g in rate)
