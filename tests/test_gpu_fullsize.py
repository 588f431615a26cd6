"""Whole-run comparisons at the benchmark sizes, in the configuration the
benchmark times (driver chosen by the library).  C4 compares a sample of batch
rows (batch rows are independent); C5 the first steps of the full network.

Strict per-step parity at these sizes is asserted along the GPU's own
trajectory (one oracle step from the GPU's state at sampled steps).  Over a
whole run two effects of float32 evaluation accumulate and are bounded here
instead:
  * rate mode: neurons with intercepts close to the radius have gains of 1e4
    to 1e5, so float32 rounding of their input moves their rate by far more
    than 1e-5 of the peak rate.  Neuron probes are checked with the
    backward-error test (exact rate of a current within 1e-4 of its term
    scale: one step holds 1e-5, but a second layer's current also carries the
    first layer's rate errors through a 1024-wide sum); decoded probes are
    held to 1e-4 relative (measured: 4.5e-5 for the circular-convolution net,
    5.9e-5 for the classifier).
  * spiking: a spike moved across threshold by rounding perturbs every
    downstream ensemble by a whole spike, so spike trains of large networks
    diverge (chaos).  Whole runs check validity (every output is 0 or
    amplitude/dt) and population rates within 2%; flips are reported."""
import numpy as np
import pytest

import paper_1805_11144_amd as M
from oracle.sim import OracleSim
from synth import make_workload
from tests.parity import flip_fraction, lif_rate_inverse_ok, rel_err, unpaired_flips

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
    probed = tuple(sorted({p.target[1] for p in w.spec.probes if p.target[0] == "neurons"}))
    ref = OracleSim(w.spec, minibatch=B, param_dtype=np.float32, record_current=probed)
    ref.run_steps(n, feeds)
    cur = {i: ref.current_data(i) for i in probed}
    return [ref.data(p) for p in range(len(w.spec.probes))], cur


def check(w, got, oracle_out, spiking):
    exp, cur = oracle_out
    for pi, (g, e) in enumerate(zip(got, exp)):
        p = w.spec.probes[pi]
        if spiking and p.target[0] == "neurons":
            f, u = flip_fraction(g, e), unpaired_flips(g, e)
            height = np.float32(w.spec.ensembles[p.target[1]].amplitude / w.spec.dt)
            ng, ne = int((g > 0).sum()), int((e > 0).sum())
            print(f"{w.name} probe {pi}: flips {f:.2e} of {ne} spikes, unpaired {u}, "
                  f"spike count {ng} vs {ne}")
            assert np.all((g == 0) | np.isclose(g, height, rtol=1e-6, atol=0))
            assert abs(ng - ne) <= 0.02 * ne
        elif not spiking and p.target[0] == "neurons" and p.synapse is None:
            ens = w.spec.ensembles[p.target[1]]
            J, S = cur[p.target[1]]
            if p.neuron_slice is not None:
                J, S = J[..., p.neuron_slice[0]:p.neuron_slice[1]], S[..., p.neuron_slice[0]:p.neuron_slice[1]]
            nf, bad5 = lif_rate_inverse_ok(g, e, J, S, ens.amplitude, ens.tau_rc, ens.tau_ref)
            _, bad = lif_rate_inverse_ok(g, e, J, S, ens.amplitude, ens.tau_rc, ens.tau_ref,
                                         rtol=1e-4)
            print(f"{w.name} probe {pi}: rel {rel_err(g, e):.2e}; {nf} elements outside the forward "
                  f"bound, {bad5} / {bad} outside the backward bound at 1e-5 / 1e-4")
            assert bad == 0
        elif not spiking:
            r = rel_err(g, e)
            print(f"{w.name} probe {pi}: rel {r:.2e}")
            assert r <= 1e-4
        else:
            print(f"{w.name} probe {pi}: abs {float(np.abs(g - e).max()):.2e} (after spike flips)")
            assert np.all(np.isfinite(g))


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
