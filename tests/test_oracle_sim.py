"""Pins for oracle/sim.py: closed forms through whole networks, brute force
against the scalar interpreter, and the minibatch / split-run invariants."""
import math

import numpy as np
import pytest

from oracle.build import build_params
from oracle.scalar import run_scalar
from oracle.sim import CycleError, OracleSim
from synth import Connection, Ensemble, ModelSpec, Node, Probe, make_workload
from synth.configs import cconv_transforms, lif_ensemble

DT = 0.001


def test_probe_lowpass_step_response():
    """Probe filter on a constant 1: y_k = 1 - a^k, exact at t = k dt."""
    m = ModelSpec(dt=DT)
    m.add_node(Node(size=1, value=np.array([1.0])))
    tau = 0.02
    m.probe(Probe(target=("node", 0), synapse=tau))
    sim = OracleSim(m)
    sim.run_steps(200)
    y = sim.data(0)[0, :, 0]
    k = np.arange(1, 201)
    np.testing.assert_allclose(y, 1.0 - np.exp(-k * DT / tau), rtol=0, atol=1e-14)


def test_connection_lowpass_impulse_response_and_delay():
    """Impulse 1/dt at step 1 through a filtered connection into a passthrough:
    the passthrough reads the filter state left by the previous step, so
    P_1 = 0 and P_k = (1 - a) a^(k-2) / dt for k >= 2."""
    m = ModelSpec(dt=DT)
    m.add_node(Node(size=1))
    m.add_node(Node(size=1, passthrough=True))
    tau = 0.01
    m.connect(Connection(pre=("node", 0), post=("node", 1), synapse=tau))
    m.probe(Probe(target=("node", 1)))
    feed = np.zeros((1, 300, 1)); feed[0, 0, 0] = 1.0 / DT
    sim = OracleSim(m)
    sim.run_steps(300, {0: feed})
    p = sim.data(0)[0, :, 0]
    a = math.exp(-DT / tau)
    k = np.arange(1, 301)
    expect = np.where(k >= 2, (1 - a) * a ** (k - 2.0) / DT, 0.0)
    np.testing.assert_allclose(p, expect, rtol=1e-12, atol=1e-12)
    # as dt -> 0 the response approaches exp(-t/tau)/tau
    assert p[1] * tau == pytest.approx(1.0, rel=0.06)


def test_integrator_ramp_direct_mode():
    """Direct-mode integrator (input transform tau, recurrent transform 1, both
    lowpass tau): represented value x_k = (1 - a) tau sum_{j<k} u_j exactly."""
    w = make_workload("c1")
    sim = OracleSim(w.spec, direct=frozenset({0}))
    u = np.random.default_rng(7).uniform(-1, 1, size=(1, 400, 1))
    sim.run_steps(400, {0: u})
    # probe 0 is a filtered decoded probe; read the represented value by a
    # second, unfiltered probe on the same ensemble
    m = w.spec
    m2 = ModelSpec(nodes=m.nodes, ensembles=m.ensembles, connections=m.connections,
                   probes=[Probe(target=("ens", 0))], dt=m.dt)
    sim = OracleSim(m2, direct=frozenset({0}))
    sim.run_steps(400, {0: u})
    x = sim.data(0)[0, :, 0]
    a = math.exp(-DT / 0.1)
    expect = (1 - a) * 0.1 * np.concatenate([[0.0], np.cumsum(u[0, :-1, 0])])
    np.testing.assert_allclose(x, expect, rtol=1e-10, atol=1e-13)
    # slope per unit input is (1 - a) tau / dt = 0.99502 per second
    assert (1 - a) * 0.1 / DT == pytest.approx(0.99502, abs=1e-5)


def test_cconv_direct_mode_equals_fft_circular_convolution():
    w = make_workload("c2", n_steps=400, minibatch=3)
    direct = frozenset(range(len(w.spec.ensembles)))
    sim = OracleSim(w.spec, minibatch=3, direct=direct)
    sim.run_steps(400, w.feeds)
    out = sim.data(0)[:, -1, :]
    a = w.feeds[0][:, 0, :].astype(np.float64)
    b = w.feeds[1][:, 0, :].astype(np.float64)
    expect = np.real(np.fft.ifft(np.fft.fft(a, axis=1) * np.fft.fft(b, axis=1), axis=1))
    np.testing.assert_allclose(out, expect, rtol=0, atol=1e-12)


def test_node_driven_ensemble_spikes_match_closed_form():
    Js = [1.2, 2.0, 5.0, 40.0]
    m = ModelSpec(dt=DT)
    m.add_ensemble(Ensemble(n_neurons=4, dims=1, encoders=np.ones((4, 1)),
                            eval_points=np.zeros((1, 1)), gains=np.ones(4),
                            biases=np.array(Js)))
    m.probe(Probe(target=("neurons", 0)))
    sim = OracleSim(m)
    sim.run_steps(2000)
    s = sim.data(0)[0]
    for i, J in enumerate(Js):
        t1 = 0.02 * math.log(J / (J - 1))
        steps = np.nonzero(s[:, i])[0] + 1
        expect = [math.ceil((t1 + j * (0.002 + t1)) / DT - 1e-9) for j in range(len(steps))]
        assert list(steps) == expect


def _three_neuron_net(w_rec, in_synapse=0.005):
    m = ModelSpec(dt=DT)
    m.add_node(Node(size=1, value=np.array([0.7])))
    m.add_ensemble(Ensemble(n_neurons=3, dims=1, encoders=np.array([[1.0], [-1.0], [1.0]]),
                            eval_points=np.zeros((1, 1)),
                            gains=np.array([2.0, 1.5, 3.0]), biases=np.array([1.1, 1.8, 0.4])))
    dec = np.array([[0.004], [-0.003], [0.002]])
    m.connect(Connection(pre=("node", 0), post=("ens", 0), transform=1.0, synapse=in_synapse))
    m.connect(Connection(pre=("ens", 0), post=("ens", 0), transform=w_rec, decoders=dec,
                         synapse=0.05))
    m.probe(Probe(target=("neurons", 0)))
    return m


def test_three_neuron_net_brute_force():
    m = _three_neuron_net(0.8)
    sim = OracleSim(m)
    sim.run_steps(600)
    ref = run_scalar(m, build_params(m), 600)
    s_vec = sim.data(0)[0]
    s_sc = np.array(ref[0][0])
    assert np.array_equal(s_vec > 0, s_sc > 0)
    np.testing.assert_allclose(s_vec, s_sc, rtol=1e-12, atol=0)


def test_three_neuron_net_without_recurrence_matches_closed_form():
    """Recurrent weight 0 and an unfiltered input: every neuron sees a constant
    J = gain * encoder * 0.7 + bias from step 1, so its spike steps are the
    closed-form ceil(t_j / dt); a neuron with J <= 1 stays silent."""
    m = _three_neuron_net(0.0, in_synapse=None)
    sim = OracleSim(m)
    sim.run_steps(1500)
    s = sim.data(0)[0]
    ref = run_scalar(m, build_params(m), 1500)
    assert np.array_equal(s > 0, np.array(ref[0][0]) > 0)
    for i, (g, e, b) in enumerate([(2.0, 1, 1.1), (1.5, -1, 1.8), (3.0, 1, 0.4)]):
        J = g * e * 0.7 + b
        steps = list(np.nonzero(s[:, i])[0] + 1)
        if J <= 1:
            assert steps == []
            continue
        t1 = 0.02 * math.log(J / (J - 1))
        expect = [math.ceil((t1 + j * (0.002 + t1)) / DT - 1e-9) for j in range(len(steps))]
        assert len(steps) > 100 and steps == expect


def _random_small_model(seed):
    rng = np.random.default_rng(seed)
    m = ModelSpec(dt=DT)
    m.add_node(Node(size=2))                                   # fed
    m.add_node(Node(size=3, passthrough=True))
    m.add_node(Node(size=1, value=np.array([0.3])))            # constant
    for i in range(3):
        m.add_ensemble(lif_ensemble(rng, 5, 2, 40, "lif" if i != 1 else "lif_rate"))
    m.connect(Connection(pre=("node", 0), post=("node", 1), transform=rng.standard_normal((3, 2)),
                         synapse=0.01))
    m.connect(Connection(pre=("node", 1), post=("ens", 0), transform=rng.standard_normal((2, 2)),
                         pre_slice=(0, 2)))
    m.connect(Connection(pre=("node", 2), post=("ens", 1), transform=1.0, post_slice=(1, 2)))
    m.connect(Connection(pre=("ens", 0), post=("ens", 1), transform=0.5, synapse=0.005))
    m.connect(Connection(pre=("ens", 1), post=("ens", 2), function="product",
                         transform=rng.standard_normal((2, 1)), synapse=None))
    m.connect(Connection(pre=("neurons", 2), post=("neurons", 0),
                         transform=0.01 * rng.standard_normal((5, 5)), synapse=0.02))
    m.connect(Connection(pre=("ens", 2), post=("node", 1), transform=rng.standard_normal((1, 2)),
                         post_slice=(2, 3), synapse=0.003))
    m.probe(Probe(target=("ens", 2), synapse=0.01))
    m.probe(Probe(target=("neurons", 0)))
    m.probe(Probe(target=("node", 1)))
    m.probe(Probe(target=("neurons", 1), neuron_slice=(1, 4)))
    return m


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_random_small_models_brute_force(seed):
    m = _random_small_model(seed)
    B, T = 2, 120
    feed = np.random.default_rng(100 + seed).uniform(-1, 1, (B, T, 2))
    sim = OracleSim(m, minibatch=B)
    sim.run_steps(T, {0: feed})
    ref = run_scalar(m, build_params(m), T, {0: feed}, minibatch=B)
    for pi in range(len(m.probes)):
        got = sim.data(pi)
        exp = np.array(ref[pi])
        np.testing.assert_allclose(got, exp, rtol=1e-10, atol=1e-10 * max(1.0, np.abs(exp).max()))


def test_minibatch_equals_sequential_runs_with_reset():
    w = make_workload("c2", n_steps=60, minibatch=4)
    sim = OracleSim(w.spec, minibatch=4)
    sim.run_steps(60, w.feeds)
    batched = sim.data(0)
    one = OracleSim(w.spec, minibatch=1)
    for b in range(4):
        one.reset()
        one.run_steps(60, {k: v[b:b + 1] for k, v in w.feeds.items()})
        np.testing.assert_allclose(one.data(0)[0], batched[b], rtol=1e-12, atol=1e-12)


def test_split_runs_equal_one_run():
    w = make_workload("c1", n_steps=300)
    a = OracleSim(w.spec); a.run_steps(300, w.feeds)
    b = OracleSim(w.spec)
    b.run_steps(100, {0: w.feeds[0][:, :100]})
    b.run_steps(200, {0: w.feeds[0][:, 100:]})
    np.testing.assert_array_equal(a.data(1), b.data(1))
    np.testing.assert_array_equal(a.data(0), b.data(0))


def test_unfiltered_cycle_is_an_error():
    m = ModelSpec(dt=DT)
    m.add_node(Node(size=1, passthrough=True))
    m.add_node(Node(size=1, passthrough=True))
    m.connect(Connection(pre=("node", 0), post=("node", 1)))
    m.connect(Connection(pre=("node", 1), post=("node", 0)))
    with pytest.raises(CycleError):
        OracleSim(m)


def test_integrator_tracks_integral_with_neurons():
    w = make_workload("c1", neuron_type="lif_rate")
    sim = OracleSim(w.spec)
    sim.run_steps(1000, w.feeds)
    x = sim.data(0)[0, :, 0]
    t = np.arange(1, 1001) * DT
    target = 0.5 / (2 * np.pi) * (1 - np.cos(2 * np.pi * t))
    assert np.sqrt(np.mean((x - target) ** 2)) < 0.05


def test_recorded_current_reproduces_rate_probe():
    """The recorded input current J gives back the rate probe through the
    closed-form rate, and the term scale bounds |J|."""
    from oracle.neurons import lif_rate
    from synth import make_workload
    w = make_workload("c2", neuron_type="lif_rate", n_steps=20, minibatch=2, n_neurons=20,
                      n_eval=100)
    sim = OracleSim(w.spec, minibatch=2, record_current=(0, 1))
    sim.run_steps(20, w.feeds)
    for pi, p in enumerate(w.spec.probes):
        if p.target[0] != "neurons":
            continue
        e = w.spec.ensembles[p.target[1]]
        J, S = sim.current_data(p.target[1])
        assert J.shape == sim.data(pi).shape
        np.testing.assert_array_equal(sim.data(pi), e.amplitude * lif_rate(J, e.tau_rc, e.tau_ref))
        assert np.all(S >= np.abs(J) * (1 - 1e-12))
        assert (J > 1).any() and (J <= 1).any()


def test_rate_backward_check_accepts_oracle_and_rejects_offsets():
    """The backward-error check passes the oracle against itself and fails a
    probe whose rates come from currents shifted well beyond the bound."""
    from oracle.neurons import lif_rate
    from synth import make_workload
    from tests.parity import lif_rate_inverse_ok
    w = make_workload("c2", neuron_type="lif_rate", n_steps=20, minibatch=2, n_neurons=20,
                      n_eval=100)
    sim = OracleSim(w.spec, minibatch=2, record_current=(0,))
    sim.run_steps(20, w.feeds)
    pi = next(i for i, p in enumerate(w.spec.probes) if p.target == ("neurons", 0))
    e = w.spec.ensembles[0]
    J, S = sim.current_data(0)
    exp = sim.data(pi)
    assert lif_rate_inverse_ok(exp, exp, J, S, e.amplitude, e.tau_rc, e.tau_ref) == (0, 0)
    off = e.amplitude * lif_rate(J + 1e-3 * S, e.tau_rc, e.tau_ref)
    nf, bad = lif_rate_inverse_ok(off, exp, J, S, e.amplitude, e.tau_rc, e.tau_ref)
    assert bad > 0


def test_relu_ensemble_matches_closed_form():
    """ReLU neurons fed by a constant node through a lowpass synapse: the
    ensemble reads the filter state left by the previous step (R4), so at step
    k (1-based) x_k = 0.7 (1 - a^(k-1)), and each output is
    amplitude * max(gain * encoder * x_k + bias, 0)."""
    gains, biases, enc = np.array([2.0, 1.5, 3.0]), np.array([0.1, -0.8, -1.5]), np.array([1.0, -1.0, 1.0])
    m = ModelSpec(dt=DT)
    m.add_node(Node(size=1, value=np.array([0.7])))
    m.add_ensemble(Ensemble(n_neurons=3, dims=1, encoders=enc[:, None], eval_points=np.zeros((1, 1)),
                            gains=gains, biases=biases, neuron_type="relu", amplitude=0.5))
    m.connect(Connection(pre=("node", 0), post=("ens", 0), transform=1.0, synapse=0.01))
    m.probe(Probe(target=("neurons", 0)))
    sim = OracleSim(m)
    sim.run_steps(50)
    a = math.exp(-DT / 0.01)
    k = np.arange(1, 51)[:, None]
    x = 0.7 * (1.0 - a ** (k - 1))
    expect = 0.5 * np.maximum(gains * enc * x + biases, 0.0)
    np.testing.assert_allclose(sim.data(0)[0], expect, rtol=1e-13, atol=1e-15)
    assert (expect[:, 2] == 0).sum() > 0 and (expect[:, 2] > 0).sum() > 0   # neuron 2 crosses 0


def test_relu_decoders_solve_the_normal_equations():
    from oracle.build import ensemble_activities, ensemble_gain_bias, ridge_decoders
    rng = np.random.default_rng(11)
    e = Ensemble(n_neurons=60, dims=2, encoders=rng.normal(size=(60, 2)), eval_points=rng.uniform(-1, 1, (300, 2)),
                 max_rates=rng.uniform(200, 400, 60), intercepts=rng.uniform(-1, 1, 60), neuron_type="relu")
    e.encoders /= np.linalg.norm(e.encoders, axis=1, keepdims=True)
    g, b = ensemble_gain_bias(e)
    A = ensemble_activities(e, g, b, e.eval_points)
    np.testing.assert_allclose(A, np.maximum((e.eval_points @ e.encoders.T) * g + b, 0.0), rtol=1e-13, atol=1e-9)
    D = ridge_decoders(A, e.eval_points, 0.1)
    lam = 300 * (0.1 * A.max()) ** 2
    resid = (A.T @ A + lam * np.eye(60)) @ D - A.T @ e.eval_points
    assert np.abs(resid).max() <= 1e-8 * np.abs(A.T @ e.eval_points).max()


def test_float32_instruments_stay_close_and_leave_the_default_alone():
    """The oracle's float32 measuring modes: arith_dtype=float32 keeps every
    state array in float32 and lands within float32 rounding of the float64
    run (rate mode, 40 steps: relative 1e-4 at most, and not bit-identical);
    current_dtype=float32 changes the float64 run only through rounded
    currents; the default float64 run is unchanged by either option's
    existence (two default runs are identical)."""
    from synth import make_workload
    w = make_workload("c2", neuron_type="lif_rate", n_steps=40, minibatch=2, n_neurons=20, n_eval=200)
    runs = {}
    for key, kw in {"f64": {}, "f64b": {}, "arith32": dict(arith_dtype=np.float32),
                    "cur32": dict(current_dtype=np.float32)}.items():
        r = OracleSim(w.spec, minibatch=w.minibatch, param_dtype=np.float32, **kw)
        r.run_steps(w.n_steps, w.feeds)
        runs[key] = (r, r.data(0))
    assert np.array_equal(runs["f64"][1], runs["f64b"][1])
    r32, d32 = runs["arith32"]
    assert all(v.dtype == np.float32 for v in r32.y.values()) and d32.dtype == np.float32
    ref = runs["f64"][1]
    for key in ("arith32", "cur32"):
        diff = np.abs(runs[key][1] - ref).max() / np.abs(ref).max()
        assert 0 < diff <= 1e-4, (key, diff)
