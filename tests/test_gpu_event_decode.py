"""Event-driven decoding (the `decode` option): the fused small-minibatch
ensemble kernel reads a neuron's decoders only when it spikes.  A silent
neuron adds exact zeros to the dense sum, so every probe must equal the dense
run's (value equality; the sign of a zero sum may differ), and through it the
oracle bounds of the dense run hold as well."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from oracle.sim import OracleSim
from synth import make_workload
from tests.parity import check_spiking_probe, float32_run

pytestmark = pytest.mark.gpu

CASES = {
    "c1": dict(n_steps=300),                                        # 1-D decoders (scalar path)
    "c2": dict(n_steps=60, minibatch=3, n_neurons=20, n_eval=200),  # product decoders, B = 3
    "c5": dict(n_steps=60, n_ens=12, n_neurons=40, n_eval=200, n_input_targets=4, n_probed=3),
}


def run(w, **opts):
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, **opts) as sim:
        sim.run_steps(w.n_steps, w.feeds)
        return [sim.data(p) for p in range(len(w.spec.probes))]


@pytest.mark.parametrize("driver", ["graph", "steps"])
@pytest.mark.parametrize("name", sorted(CASES))
def test_event_decode_equals_dense(name, driver):
    drv = {"graph": M.DRIVER_GRAPH, "steps": M.DRIVER_STEPS}[driver]
    w = make_workload(name, neuron_type="lif", **CASES[name])
    dense = run(w, driver=drv)
    event = run(w, driver=drv, decode="event")
    for pi, (a, b) in enumerate(zip(dense, event)):
        assert np.array_equal(a, b), (name, driver, pi, float(np.abs(a - b).max()))
    ref = OracleSim(w.spec, minibatch=w.minibatch, param_dtype=np.float32)
    ref.run_steps(w.n_steps, w.feeds)
    f32 = float32_run(w.spec, w.minibatch, w.n_steps, w.feeds)
    for pi, g in enumerate(event):
        check_spiking_probe(f"{name} {driver} probe {pi}", w.spec.probes[pi], g, ref.data(pi), f32[pi])


def test_event_decode_rate_mode_is_dense():
    """Rate neurons are not spike-sparse: the option leaves them dense."""
    w = make_workload("c5", neuron_type="lif_rate", **CASES["c5"])
    a, b = run(w, driver=M.DRIVER_GRAPH), run(w, driver=M.DRIVER_GRAPH, decode="event")
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.timeout(300)
def test_event_decode_c5_full_width():
    """The full C5 width (5000 ensembles x 500 neurons, 16-D) for 60 steps in
    the benchmark's launch configuration: equal to dense decoding."""
    w = make_workload("c5", n_steps=60)
    a = run(w, unroll=20, probe_capacity_steps=60)
    b = run(w, unroll=20, probe_capacity_steps=60, decode="event")
    for pi, (x, y) in enumerate(zip(a, b)):
        assert np.array_equal(x, y), (pi, float(np.abs(x - y).max()))


def test_event_decode_rejects_unknown_value():
    w = make_workload("c1", n_steps=5)
    with pytest.raises(M.MergesimError):
        M.Simulator(M.model_from_spec(w.spec), decode=7)
