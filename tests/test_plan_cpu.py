"""CPU tests of the library's host side (no GPU): the double-precision build
step against the oracle's, and the merged plan executed in float64 against the
unmerged oracle."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from oracle.build import build_params
from oracle.sim import OracleSim
from synth import make_workload
from tests.plan_exec import PlanExecutor

SMALL = {
    "c1": dict(n_steps=200),
    "c2": dict(n_steps=60, minibatch=3, n_neurons=20, n_eval=200),
    "c3": dict(n_steps=30, minibatch=4, n_hidden=96, n_in=50),
    "c4": dict(n_steps=60, minibatch=3, n_ens=6, n_neurons=40, n_eval=200),
    "c5": dict(n_steps=40, n_ens=12, n_neurons=40, n_eval=200, n_input_targets=4, n_probed=3),
    "bg": dict(n_steps=60, minibatch=2, D=6, n_neurons=20, n_eval=100),
}


@pytest.mark.parametrize("neuron_type", ["lif", "relu", "softlif_rate"])
@pytest.mark.parametrize("name", ["c1", "c2", "c4", "c5", "bg"])
def test_build_params_match_oracle(name, neuron_type):
    w = make_workload(name, neuron_type=neuron_type, **SMALL[name])
    plan = M.Plan(M.model_from_spec(w.spec), minibatch=w.minibatch)
    P = build_params(w.spec)
    for e in range(len(w.spec.ensembles)):
        np.testing.assert_allclose(plan.param(M.mergesim.PARAM_GAIN, e), P.gain[e], rtol=1e-12)
        np.testing.assert_allclose(plan.param(M.mergesim.PARAM_BIAS, e), P.bias[e], rtol=1e-12,
                                   atol=1e-12 * np.abs(P.bias[e]).max())
    for (e, fn), D in P.decoders.items():
        got = plan.param(M.mergesim.PARAM_DECODERS, e, 1 if fn == "product" else 0).reshape(D.shape)
        np.testing.assert_allclose(got, D, rtol=1e-6, atol=1e-9 * np.abs(D).max())


@pytest.mark.parametrize("name", list(SMALL))
@pytest.mark.parametrize("neuron_type", ["lif_rate", "lif", "relu", "softlif_rate"])
@pytest.mark.parametrize("opts", [dict(), dict(planner=M.PLANNER_GREEDY), dict(sort=False),
                                  dict(simplify=False), dict(merge=False), dict(fuse=False)])
def test_plan_execution_matches_oracle(name, neuron_type, opts):
    w = make_workload(name, neuron_type=neuron_type, **SMALL[name])
    plan = M.Plan(M.model_from_spec(w.spec), minibatch=w.minibatch, **opts)
    ref = OracleSim(w.spec, minibatch=w.minibatch, param_dtype=np.float32)
    ex = PlanExecutor(plan, w.spec, w.minibatch, params_from=ref)
    ex.run(w.n_steps, w.feeds)
    ref.run_steps(w.n_steps, w.feeds)
    for pi in range(len(w.spec.probes)):
        got, exp = ex.data(pi), ref.data(pi)
        assert got.shape == exp.shape
        scale = max(1.0, np.abs(exp).max())
        if neuron_type == "lif" and w.spec.probes[pi].target[0] == "neurons":
            assert np.array_equal(got > 0, exp > 0)
        np.testing.assert_allclose(got, exp, rtol=0, atol=1e-11 * scale)
