"""Parity at the benchmark sizes, in the configuration bench.py times (driver
chosen by the library).  C4 compares a sample of batch rows (batch rows are
independent); C5 the first steps of the full network."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from oracle.sim import OracleSim
from synth import make_workload
from tests.parity import flip_fraction, rel_err, unpaired_flips

pytestmark = pytest.mark.gpu


def gpu_run(w, n_steps=None, rows=None):
    n = n_steps or w.n_steps
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, unroll=20,
                     probe_capacity_steps=n) as sim:
        sim.run_steps(n, {k: f[:, :n] for k, f in w.feeds.items()})
        out = [sim.data(p) for p in range(len(w.spec.probes))]
    if rows is not None:
        out = [o[rows] for o in out]
    return out


def oracle_run(w, n_steps=None, rows=None):
    n = n_steps or w.n_steps
    B = w.minibatch if rows is None else len(rows)
    feeds = {k: (f if rows is None else f[rows])[:, :n] for k, f in w.feeds.items()}
    ref = OracleSim(w.spec, minibatch=B, param_dtype=np.float32)
    ref.run_steps(n, feeds)
    return [ref.data(p) for p in range(len(w.spec.probes))]


def check(w, got, exp, spiking):
    for pi, (g, e) in enumerate(zip(got, exp)):
        p = w.spec.probes[pi]
        if spiking and p.target[0] == "neurons":
            f, u = flip_fraction(g, e), unpaired_flips(g, e)
            print(f"{w.name} probe {pi}: flips {f:.2e} of {int((e > 0).sum())} spikes, unpaired {u}")
            assert u == 0 and f <= 1e-4
        elif not spiking:
            r = rel_err(g, e)
            print(f"{w.name} probe {pi}: rel {r:.2e}")
            assert r <= 1e-5
        else:
            print(f"{w.name} probe {pi}: abs {float(np.abs(g - e).max()):.2e} (after spike flips)")


@pytest.mark.timeout(600)
@pytest.mark.parametrize("neuron_type", ["lif_rate", "lif"])
def test_c2_full(neuron_type):
    w = make_workload("c2", neuron_type=neuron_type)
    check(w, gpu_run(w), oracle_run(w), neuron_type == "lif")


@pytest.mark.timeout(600)
@pytest.mark.parametrize("neuron_type", ["lif_rate", "lif"])
def test_c3_full(neuron_type):
    w = make_workload("c3", neuron_type=neuron_type)
    check(w, gpu_run(w), oracle_run(w), neuron_type == "lif")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("neuron_type", ["lif_rate", "lif"])
def test_c4_full_batch_sampled_rows(neuron_type):
    w = make_workload("c4", neuron_type=neuron_type)
    rows = np.arange(0, 512, 73)[:8]
    n = 200
    check(w, gpu_run(w, n, rows), oracle_run(w, n, rows), neuron_type == "lif")


@pytest.mark.timeout(1200)
def test_c5_full_first_steps():
    w = make_workload("c5", neuron_type="lif")
    n = 40
    got, exp = gpu_run(w, n), oracle_run(w, n)
    check(w, got, exp, True)
