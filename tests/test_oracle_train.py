"""Pins of the training oracle (oracle/train.py; paper Sec. 3.2: an objective
on probe outputs minimised by gradient descent through the unrolled steps).

  * its forward pass equals OracleSim's probe data (an independent numpy
    stepper) on the three training shapes;
  * every gradient equals central finite differences of the objective as
    OracleSim computes it (numpy, no automatic differentiation): a dropped
    term, a wrong sign, a transposed operand or a missed step of the filter
    recursion changes some gradient entry by far more than the bound;
  * two models small enough to differentiate by hand: one ReLU neuron for one
    step, and a node feeding a passthrough node through a scalar transform and
    a lowpass synapse over several steps (the delay and the geometric
    impulse response of the filter enter the gradient).
"""
import math

import numpy as np
import pytest

from oracle.sim import OracleSim
from oracle.train import TrainOracle, objective_numpy, trainable_params
from synth import Connection, Ensemble, ModelSpec, Node, Probe, make_train

SHAPES = {
    "mlp": dict(n_steps=6, minibatch=2, n_in=5, n_hidden=12, n_out=3),
    "chain": dict(n_steps=6, minibatch=2, n_ens=3, n_neurons=10, dims=2, n_eval=40),
    "cconv": dict(n_steps=5, minibatch=2, D=4, n_neurons=8, n_eval=40),
}


def _small(kind, neuron_type):
    """A small training model; intercepts drawn from [-0.9, 0.9] so that no
    current sits exactly on a kink of the rate curves (the classifier's
    default intercept 0 with zero filter states puts ReLU currents at exactly
    0, where a central difference straddles the kink)."""
    w, targets = make_train(kind, neuron_type=neuron_type, **SHAPES[kind])
    rng = np.random.default_rng(5)
    for e in w.spec.ensembles:
        e.intercepts = rng.uniform(-0.9, 0.9, e.n_neurons)
    return w, targets


@pytest.mark.parametrize("neuron_type", ["lif_rate", "softlif_rate", "relu"])
@pytest.mark.parametrize("kind", list(SHAPES))
def test_forward_equals_oracle_sim(kind, neuron_type):
    w, targets = _small(kind, neuron_type)
    tr = TrainOracle(w.spec, w.minibatch)
    _, _, probes = tr.loss_and_grads(w.n_steps, w.feeds, targets)
    ref = OracleSim(w.spec, minibatch=w.minibatch, param_dtype=np.float32)
    ref.run_steps(w.n_steps, w.feeds)
    for pi in range(len(w.spec.probes)):
        exp = ref.data(pi)
        np.testing.assert_allclose(probes[pi], exp, rtol=0, atol=1e-12 * max(1.0, np.abs(exp).max()))
    loss = objective_numpy(w.spec, w.minibatch, w.n_steps, w.feeds, targets, tr.params)
    got, _, _ = tr.loss_and_grads(w.n_steps, w.feeds, targets)
    assert got == pytest.approx(loss, rel=1e-12)


def _fd_check(w, targets, tr, per_tensor=5, seed=0, h_rel=1e-6):
    """Central differences of objective_numpy at a few entries of every
    trained tensor against the oracle's gradient."""
    loss, grads, _ = tr.loss_and_grads(w.n_steps, w.feeds, targets)
    rng = np.random.default_rng(seed)
    checked = 0
    for key, val in tr.params.items():
        g = grads[key]
        scale = max(np.abs(g).max(), 1e-12)
        flat = np.arange(val.size)
        picks = rng.choice(flat, size=min(per_tensor, val.size), replace=False)
        # the largest entry too, so that every tensor is checked where it matters
        picks = np.unique(np.append(picks, np.argmax(np.abs(g).ravel())))
        # steps relative to the tensor's size (decoders are ~1e-3), so that
        # the truncation error (h^2 times the third derivative) stays small
        size = max(np.abs(val).max(), 1e-6)
        for i in picks:
            h = h_rel * size
            # rounding of the two objective values: about eps |L| / h
            noise = 1e-15 * abs(loss) / h
            P = {k: v.copy() for k, v in tr.params.items()}
            P[key].flat[i] = val.flat[i] + h
            lp = objective_numpy(w.spec, w.minibatch, w.n_steps, w.feeds, targets, P)
            P[key].flat[i] = val.flat[i] - h
            lm = objective_numpy(w.spec, w.minibatch, w.n_steps, w.feeds, targets, P)
            fd = (lp - lm) / (2 * h)
            assert abs(fd - g.flat[i]) <= 1e-6 * scale + noise, (key, int(i), fd, g.flat[i], scale)
            checked += 1
    return checked


@pytest.mark.parametrize("neuron_type", ["lif_rate", "softlif_rate", "relu"])
@pytest.mark.parametrize("kind", list(SHAPES))
def test_gradients_equal_finite_differences(kind, neuron_type):
    w, targets = _small(kind, neuron_type)
    tr = TrainOracle(w.spec, w.minibatch)
    kinds = {k[0] for k in tr.params}
    # every kind of trained parameter the shape has is present and checked
    expect = {"mlp": {"bias", "T"}, "chain": {"enc", "bias", "dec", "T"},
              "cconv": {"enc", "bias", "dec", "T"}}[kind]
    assert expect <= kinds
    assert _fd_check(w, targets, tr) >= 3 * len(tr.params)


def test_gradients_after_descent_steps_equal_finite_differences():
    """The pins hold away from the initial parameters too (after two steps of
    gradient descent, where no gradient is near zero by construction)."""
    w, targets = _small("chain", "lif_rate")
    tr = TrainOracle(w.spec, w.minibatch)
    for _ in range(2):
        _, g, _ = tr.loss_and_grads(w.n_steps, w.feeds, targets)
        tr.sgd(g, 1e-3)
    _fd_check(w, targets, tr, seed=1)


def test_one_relu_neuron_by_hand():
    """J = b + e x, s = J (ReLU, amplitude 1), p = d s, L = (p - t)^2 for one
    step: with x = 0.5, e = 2, b = 0.25, d = 0.8, t = 0.3 the probe is 1.0,
    L = 0.49, dL/dd = 2 (p - t) s = 1.75, dL/db = 2 (p - t) d = 1.12,
    dL/de = 2 (p - t) d x = 0.56."""
    m = ModelSpec(dt=0.001)
    inp = m.add_node(Node(size=1))
    e = m.add_ensemble(Ensemble(n_neurons=1, dims=1, encoders=np.ones((1, 1)), eval_points=np.zeros((1, 1)),
                                gains=np.array([2.0]), biases=np.array([0.25]), neuron_type="relu"))
    out = m.add_node(Node(size=1, passthrough=True))
    m.connect(Connection(pre=inp, post=("ens", e)))
    m.connect(Connection(pre=("ens", e), post=out, decoders=np.array([[0.8]])))
    m.probe(Probe(target=out))
    tr = TrainOracle(m, minibatch=1, param_dtype=np.float64)
    loss, g, probes = tr.loss_and_grads(1, {0: np.full((1, 1, 1), 0.5)}, {0: np.full((1, 1, 1), 0.3)})
    assert probes[0][0, 0, 0] == pytest.approx(1.0, rel=1e-12)
    assert loss == pytest.approx(0.49, rel=1e-12)
    assert g[("cdec", 1)][0, 0] == pytest.approx(1.75, rel=1e-12)
    assert g[("bias", 0)][0] == pytest.approx(1.12, rel=1e-12)
    assert g[("enc", 0)][0, 0] == pytest.approx(0.56, rel=1e-12)
    assert g[("T", 1)][0] == pytest.approx(1.75 * 0.8 / 1.0, rel=1e-12)   # p = T d s: dL/dT = 2 (p - t) d s
    assert g[("T", 0)][0] == pytest.approx(1.12, rel=1e-12)   # x = T u: dL/dT = dL/dJ e u = 1.12 * 2 * 0.5


def test_relu_derivative_at_zero_current_is_zero():
    """The reading at the kink: a ReLU neuron whose current is exactly 0
    (zero bias, zero input) passes no gradient to its bias, while one step
    later with current 0.5 it passes d (p - t) * 2 / T (T = 2 steps)."""
    m = ModelSpec(dt=0.001)
    inp = m.add_node(Node(size=1))
    e = m.add_ensemble(Ensemble(n_neurons=1, dims=1, encoders=np.ones((1, 1)), eval_points=np.zeros((1, 1)),
                                gains=np.array([1.0]), biases=np.array([0.0]), neuron_type="relu"))
    out = m.add_node(Node(size=1, passthrough=True))
    m.connect(Connection(pre=inp, post=("ens", e)))
    m.connect(Connection(pre=("ens", e), post=out, decoders=np.array([[0.8]])))
    m.probe(Probe(target=out))
    tr = TrainOracle(m, minibatch=1, param_dtype=np.float64)
    feed = np.array([[[0.0], [0.5]]])   # J = 0, then J = 0.5
    _, g, probes = tr.loss_and_grads(2, {0: feed}, {0: np.full((1, 2, 1), 0.3)})
    assert probes[0][0, :, 0] == pytest.approx([0.0, 0.4], abs=1e-15)
    # only step 1 contributes: dL/db = (2/2) (0.4 - 0.3) * 0.8
    assert g[("bias", 0)][0] == pytest.approx(0.08, rel=1e-12)


def test_filtered_scalar_connection_by_hand():
    """u (constant 1) -> passthrough node through transform w and a lowpass
    with coefficient a: the filter state after step k is
    y_k = w (1 - a^(k+1)) and the node reads the state left by the previous
    step, so p_0 = 0 and p_k = w (1 - a^k).  L = mean_k (p_k - c)^2, hence
    dL/dw = (2/T) sum_k (w q_k - c) q_k with q_k = 1 - a^k."""
    tau, dt, T, wv, c = 0.01, 0.001, 7, 1.5, 0.4
    m = ModelSpec(dt=dt)
    inp = m.add_node(Node(size=1))
    out = m.add_node(Node(size=1, passthrough=True))
    m.connect(Connection(pre=inp, post=out, transform=wv, synapse=tau))
    m.probe(Probe(target=out))
    tr = TrainOracle(m, minibatch=1, param_dtype=np.float64)
    loss, g, probes = tr.loss_and_grads(T, {0: np.ones((1, T, 1))}, {0: np.full((1, T, 1), c)})
    a = math.exp(-dt / tau)
    q = np.array([1 - a ** k for k in range(T)])
    np.testing.assert_allclose(probes[0][0, :, 0], wv * q, rtol=1e-12, atol=1e-15)
    assert loss == pytest.approx(np.mean((wv * q - c) ** 2), rel=1e-12)
    assert g[("T", 0)][0] == pytest.approx(2.0 / T * np.sum((wv * q - c) * q), rel=1e-12)


def test_spiking_and_learning_models_are_refused():
    w, _ = make_train("mlp", neuron_type="lif", **SHAPES["mlp"])
    with pytest.raises(ValueError):
        trainable_params(OracleSim(w.spec, minibatch=1))
