"""Pins for the oracle's PES learning rule (paper Sec. 5.1, the pes benchmark:
an ensemble's output weights learn online by Prescribed Error Sensitivity;
Fig. 7's caption: one weight matrix per batch element).

The rule's step is a reading (decoders D^b <- D^b - (kappa dt / n)
outer(a^b, e^b), a the pre activity filter's state as left by the previous
step); these tests fix it from outside the oracle's code:

  * closed forms: n identical ReLU neurons of constant rate r decoding into a
    passthrough node, error = output - target.  The decoded sum S = sum_i d_i
    obeys S <- S - kappa dt r e with e = r S - t, so the output approaches the
    target geometrically with ratio 1 - kappa dt r^2 (independent of n: pins
    the 1/n scaling), and with a pre filter the ratio of step k is
    1 - kappa dt r^2 (1 - p^(k-1));
  * brute force: two neurons of different rates, two dimensions, filtered
    error connections, written out with scalar loops in this file;
  * per-row learning: each batch row learns its own target, equals a
    one-row run, and the rows' decoders differ;
  * kappa = 0 reduces to the plain decoded connection."""
import math

import numpy as np
import pytest

from oracle.sim import OracleSim
from synth import Connection, Ensemble, ModelSpec, Node, Probe
from synth.spec import PES

DT = 0.001


def _relu_ens(rates):
    n = len(rates)
    return Ensemble(n_neurons=n, dims=1, encoders=np.ones((n, 1)), eval_points=np.zeros((1, 1)),
                    gains=np.ones(n), biases=np.asarray(rates, np.float64), neuron_type="relu")


def _learner(rates, d0, kappa, pre_synapse, err_synapse=None, target=None, dims=1, synapse=None):
    """Constant-rate ReLU ensemble -> passthrough node (learned connection,
    lowpass `synapse` or none); error = node output - target, both into the
    rule.  Probe 0: the node."""
    m = ModelSpec(dt=DT)
    e = m.add_ensemble(_relu_ens(rates))
    m.ensembles[e].dims = dims
    m.ensembles[e].encoders = np.ones((len(rates), dims)) / math.sqrt(dims)
    m.ensembles[e].eval_points = np.zeros((1, dims))
    post = m.add_node(Node(size=dims, passthrough=True))
    tgt = m.add_node(Node(size=dims, value=None if target is None else np.asarray(target, np.float64)))
    c = m.connect(Connection(pre=("ens", e), post=post, decoders=np.asarray(d0, np.float64).reshape(len(rates), dims),
                             synapse=synapse, learning_rule=PES(learning_rate=kappa, pre_synapse=pre_synapse)))
    m.connect(Connection(pre=post, post=("learning", c), synapse=err_synapse))
    m.connect(Connection(pre=tgt, post=("learning", c), transform=-1.0, synapse=err_synapse))
    m.probe(Probe(target=post))
    return m, c


@pytest.mark.parametrize("n", [1, 4])
def test_unfiltered_rule_converges_geometrically(n):
    r, t, kappa, K = 50.0, 0.7, 0.02, 60
    d0 = np.full(n, 0.3 / (n * r))                  # initial output 0.3
    m, _ = _learner([r] * n, d0, kappa, None, target=[t])
    sim = OracleSim(m)
    sim.run_steps(K)
    out = sim.data(0)[0, :, 0]
    k = np.arange(1, K + 1)
    ratio = 1.0 - kappa * DT * r * r                 # 0.95
    expect = t + (0.3 - t) * ratio ** (k - 1.0)
    np.testing.assert_allclose(out, expect, rtol=0, atol=1e-13)
    # every neuron's decoder moved by the same amount
    W = sim.W[0][0, :, 0]
    np.testing.assert_allclose(W, W[0], rtol=0, atol=1e-15)


def test_pre_filtered_activity_closed_form():
    r, t, kappa, K, tau = 40.0, -0.5, 0.05, 80, 0.01
    p = math.exp(-DT / tau)
    m, _ = _learner([r] * 3, np.full(3, 0.2 / (3 * r)), kappa, tau, target=[t])
    sim = OracleSim(m)
    sim.run_steps(K)
    out = sim.data(0)[0, :, 0]
    dev, expect = 0.2 - t, []
    for k in range(1, K + 1):
        expect.append(t + dev)                      # output of step k uses the decoders before its change
        abar = r * (1.0 - p ** (k - 1))             # filter state left by step k-1
        dev *= 1.0 - kappa * DT * r * abar
    np.testing.assert_allclose(out, expect, rtol=0, atol=1e-13)
    assert out[0] == pytest.approx(0.2, abs=1e-15) and out[1] == pytest.approx(0.2, abs=1e-15)
    np.testing.assert_allclose(sim.abar[0][0], r * (1.0 - p ** K), rtol=1e-13)


@pytest.mark.parametrize("tau_l", [None, 0.004])
def test_brute_force_two_neurons_two_dims_filtered_error(tau_l):
    """Scalar loops: rates r_i, decoders d[i][j], filtered error connections
    (state from the previous step), pre filter, the learned connection
    unfiltered or filtered (its filter takes the decoders from before the
    step's change); the same definition written element by element."""
    rates, kappa, tau_e, tau_p, K = [30.0, 70.0], 0.03, 0.005, 0.02, 50
    target = [0.4, -0.25]
    d0 = [[0.001, -0.002], [0.003, 0.0005]]
    m, _ = _learner(rates, d0, kappa, tau_p, err_synapse=tau_e, target=target, dims=2, synapse=tau_l)
    sim = OracleSim(m)
    sim.run_steps(K)
    ae, ap = math.exp(-DT / tau_e), math.exp(-DT / tau_p)
    al = math.exp(-DT / tau_l) if tau_l else 0.0
    d = [row[:] for row in d0]
    ye_post, ye_tgt, abar, yl = [0.0, 0.0], [0.0, 0.0], [0.0, 0.0], [0.0, 0.0]
    outs = []
    for _ in range(K):
        dec = [sum(rates[i] * d[i][j] for i in range(2)) for j in range(2)]
        out = yl[:] if tau_l else dec                         # the passthrough node's value
        outs.append(out)
        err = [ye_post[j] + ye_tgt[j] for j in range(2)]      # filtered: previous step's states
        act = abar[:]
        for j in range(2):
            ye_post[j] = ae * ye_post[j] + (1 - ae) * out[j]
            ye_tgt[j] = ae * ye_tgt[j] + (1 - ae) * (-target[j])
            yl[j] = al * yl[j] + (1 - al) * dec[j]
        for i in range(2):
            for j in range(2):
                d[i][j] -= kappa * DT / 2 * act[i] * err[j]
            abar[i] = ap * abar[i] + (1 - ap) * rates[i]
    np.testing.assert_allclose(sim.data(0)[0], np.array(outs), rtol=0, atol=1e-14)
    np.testing.assert_allclose(sim.W[0][0], np.array(d), rtol=0, atol=1e-16)
    # learning reduced the error
    assert np.abs(np.array(outs[-1]) - target).max() < 0.5 * np.abs(np.array(outs[1]) - target).max()


def test_each_batch_row_learns_its_own_weights():
    rates, K = [20.0, 45.0, 60.0], 120
    m, c = _learner(rates, np.zeros(3), 0.02, 0.005)
    targets = np.array([[0.5], [-0.3], [0.1]])
    feed = np.broadcast_to(targets[:, None, :], (3, K, 1)).copy()
    sim = OracleSim(m, minibatch=3)
    sim.run_steps(K, {1: feed})
    for b in range(3):
        one = OracleSim(m, minibatch=1)
        one.run_steps(K, {1: feed[b:b + 1]})
        np.testing.assert_allclose(one.data(0)[0], sim.data(0)[b], rtol=0, atol=1e-14)
        np.testing.assert_allclose(one.W[c][0], sim.W[c][b], rtol=0, atol=1e-16)
    W = sim.W[c]
    assert np.abs(W[0] - W[1]).max() > 1e-4 and np.abs(W[1] - W[2]).max() > 1e-4
    # each row's output moved toward its own target
    d = sim.data(0)[:, :, 0]
    assert np.all(np.abs(d[:, -1] - targets[:, 0]) < 0.5 * np.abs(d[:, 0] - targets[:, 0]))


def test_zero_learning_rate_is_the_plain_connection():
    rates = [10.0, 35.0]
    d0 = [[0.01], [0.02]]
    m, _ = _learner(rates, d0, 0.0, 0.005, target=[1.0])
    plain = ModelSpec(dt=DT)
    e = plain.add_ensemble(_relu_ens(rates))
    post = plain.add_node(Node(size=1, passthrough=True))
    plain.connect(Connection(pre=("ens", e), post=post, decoders=np.array(d0)))
    plain.probe(Probe(target=post))
    a, b = OracleSim(m), OracleSim(plain)
    a.run_steps(30)
    b.run_steps(30)
    np.testing.assert_array_equal(a.data(0), b.data(0))


def test_error_into_a_connection_without_rule_is_rejected():
    m = ModelSpec(dt=DT)
    e = m.add_ensemble(_relu_ens([10.0]))
    post = m.add_node(Node(size=1, passthrough=True))
    c = m.connect(Connection(pre=("ens", e), post=post, decoders=np.ones((1, 1))))
    m.connect(Connection(pre=post, post=("learning", c)))
    with pytest.raises(ValueError):
        OracleSim(m)
