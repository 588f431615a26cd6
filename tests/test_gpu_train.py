"""GPU: training by gradient descent through the unrolled simulation (paper
Sec. 3.2) through the C ABI (ms_sim_train_step, ms_sim_train_param), against
the training oracle (oracle/train.py, pinned in test_oracle_train.py).

Compared element by element: the objective, every trained parameter's
gradient, the parameters after several gradient-descent steps and the probes
the training run records.  Bounds, as for every rate-mode quantity
(tests/parity.py): relative to the tensor's largest entry, within RATE_REL
(1e-5) or FLOOR_FACTOR (2) times what float32 arithmetic alone does to the
same quantity, whichever is larger.  That float32 floor is the largest
deviation from the float64 oracle among float32 runs of the oracle (which
also stores the trained parameters in float32): one with the products summed
as the CPU library sums them, one summed over slices of 16 of the inner
index in order, as the GPU's product kernels do (two equally valid float32
roundings of the same computation).

Neuron types: the smoothed LIF rate (the training stand-in for the spiking
LIF) and ReLU, whose gradients float32 computes to ~1e-6.  The exact LIF
rate's slope grows without bound at threshold, so rounding a near-threshold
current moves its derivative arbitrarily far (float32 moves the classifier's
gradients by 1e-2); its derivative is checked on a model whose neurons all
stay above threshold.

Shapes: each of the three training models at a few sizes with ragged tiles
(products of 70 -> 200 and 200 -> 200 run on the 128 x 128 weight-gradient
tiles; odd minibatches use the small-block kernels), and the 784-1024-1024-10
classifier at the benchmark's size and launch configuration (minibatch 256,
50 steps)."""
import numpy as np
import pytest
import torch

import paper_1805_11144_amd as M
from oracle.train import TrainOracle
from synth import make_train
from tests.parity import FLOOR_FACTOR, RATE_REL, rel_err

pytestmark = pytest.mark.gpu

MS = M.mergesim
TRAIN = dict(driver=M.DRIVER_WINDOW, fuse=False, simplify=False)


def _abi_key(key):
    """Oracle parameter key -> (which, id, function) of ms_sim_train_param."""
    if key[0] == "enc":
        return MS.TRAIN_ENCODERS, key[1], 0
    if key[0] == "bias":
        return MS.TRAIN_BIASES, key[1], 0
    if key[0] == "dec":
        return MS.TRAIN_DECODERS, key[1], key[2]
    if key[0] == "cdec":
        return MS.TRAIN_CONN_DECODERS, key[1], 0
    return MS.TRAIN_TRANSFORM, key[1], 0


def _gpu(w, targets, lr=0.0, steps=1, keys=()):
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, probe_capacity_steps=w.n_steps,
                     **TRAIN) as sim:
        losses = [sim.train_step(w.n_steps, w.feeds, targets, lr) for _ in range(steps)]
        grads = {k: sim.train_param(*_abi_key(k), gradient=True) for k in keys}
        params = {k: sim.train_param(*_abi_key(k)) for k in keys}
        probes = [sim.data(p) for p in range(len(w.spec.probes))]
    return losses, grads, params, probes


def _check(tag, got, exp, f32_runs, failed):
    r, floor = rel_err(got, exp), max(rel_err(f, exp) for f in f32_runs)
    bound = max(RATE_REL, FLOOR_FACTOR * floor)
    print(f"{tag}: rel {r:.2e} (float32 floor {floor:.2e}, bound {bound:.2e})")
    if not r <= bound:
        failed.append((tag, r, bound))


def _compare(w, targets, tag, lr=0.0, steps=1):
    ref = TrainOracle(w.spec, w.minibatch)
    f32 = [(TrainOracle(w.spec, w.minibatch, arith=torch.float32, chunk=ch), w.feeds) for ch in (0, 16)]
    keys = list(ref.params)
    p0 = {k: v.copy() for k, v in ref.params.items()}
    losses, grads, params, probes = _gpu(w, targets, lr, steps, keys)
    exp_losses, failed = [], []
    for it in range(steps):
        le, ge, pe = ref.loss_and_grads(w.n_steps, w.feeds, targets)
        runs = [o.loss_and_grads(w.n_steps, fd, targets) for o, fd in f32]
        exp_losses.append(le)
        _check(f"{tag} objective, step {it}", [losses[it]], [le], [[r[0]] for r in runs], failed)
        if it + 1 < steps:
            ref.sgd(ge, lr)
            for (o, _), r in zip(f32, runs):
                o.sgd(r[1], lr)
    for k in keys:   # gradients of the last step
        shape = ref.params[k].shape
        _check(f"{tag} gradient {k}", grads[k].reshape(shape), ge[k], [r[1][k] for r in runs], failed)
    if lr:
        ref.sgd(ge, lr)
        for (o, _), r in zip(f32, runs):
            o.sgd(r[1], lr)
        for k in keys:   # what the updates changed
            shape = ref.params[k].shape
            _check(f"{tag} change of {k} over {steps} steps", params[k].reshape(shape) - p0[k],
                   ref.params[k] - p0[k], [o.params[k] - p0[k] for o, _ in f32], failed)
    for pi in range(len(w.spec.probes)):   # the last step's forward run
        _check(f"{tag} probe {pi}", probes[pi], pe[pi], [r[2][pi] for r in runs], failed)
    assert not failed, failed
    return losses, exp_losses


@pytest.mark.parametrize("neuron_type", ["softlif_rate", "relu"])
@pytest.mark.parametrize("kind,kw", [
    ("mlp", dict(n_steps=12, minibatch=8, n_in=70, n_hidden=200, n_out=10)),
    ("mlp", dict(n_steps=7, minibatch=3, n_in=9, n_hidden=33, n_out=4)),
    ("chain", dict(n_steps=12, minibatch=8, n_ens=3, n_neurons=90, dims=5, n_eval=100)),
    ("chain", dict(n_steps=9, minibatch=5, n_ens=2, n_neurons=70, dims=16, n_eval=100)),
    ("cconv", dict(n_steps=10, minibatch=4, D=8, n_neurons=30, n_eval=100)),
])
def test_gradients_match_oracle(kind, kw, neuron_type):
    w, targets = make_train(kind, neuron_type=neuron_type, **kw)
    _compare(w, targets, f"{kind} {neuron_type} B={w.minibatch} T={w.n_steps}")


@pytest.mark.parametrize("kind,kw", [
    ("chain", dict(n_steps=12, minibatch=8, n_ens=3, n_neurons=90, dims=5, n_eval=100)),
    ("chain", dict(n_steps=9, minibatch=5, n_ens=2, n_neurons=70, dims=16, n_eval=100)),
])
def test_exact_lif_rate_gradients_above_threshold(kind, kw):
    """The exact LIF rate curve's derivative, on chains whose neurons all fire:
    intercepts in [-1, -0.6] and represented values of norm at most about 0.5
    keep every current at least 0.1 gain above threshold."""
    w, targets = make_train(kind, neuron_type="lif_rate", **kw)
    rng = np.random.default_rng(11)
    for e in w.spec.ensembles:
        e.intercepts = rng.uniform(-1.0, -0.6, e.n_neurons)
    _compare(w, targets, f"{kind} exact LIF rate above threshold B={w.minibatch} T={w.n_steps}")


@pytest.mark.parametrize("kind,kw", [
    ("mlp", dict(n_steps=10, minibatch=8, n_in=40, n_hidden=96, n_out=6)),
    ("chain", dict(n_steps=10, minibatch=4, n_ens=2, n_neurons=60, dims=4, n_eval=100)),
])
def test_descent_steps_match_oracle(kind, kw):
    """Three steps of gradient descent: objectives, last gradients and the
    parameters after the updates; the objective goes down."""
    w, targets = make_train(kind, **kw)
    lr = {"mlp": 2e-2, "chain": 1e-6}[kind]   # the chain's decoder gradients are ~10^4 times its decoders
    losses, exp = _compare(w, targets, f"{kind} descent", lr=lr, steps=3)
    assert losses[-1] < losses[0] and exp[-1] < exp[0]


def test_parameters_round_trip_and_restart_from_the_initial_state():
    """ms_sim_set_train_param writes what ms_sim_train_param reads (the
    decoders in the caller's [n][d] layout); a training step always starts
    from the initial state, so two steps without an update agree exactly."""
    w, targets = make_train("chain", neuron_type="relu", n_steps=6, minibatch=4, n_ens=2, n_neurons=40, dims=3,
                            n_eval=60)
    ref = TrainOracle(w.spec, w.minibatch)
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, **TRAIN) as sim:
        for k, v in ref.params.items():
            np.testing.assert_array_equal(sim.train_param(*_abi_key(k)).reshape(v.shape), v.astype(np.float32))
        l0 = sim.train_step(w.n_steps, w.feeds, targets)
        g0 = sim.train_param(MS.TRAIN_DECODERS, 1, gradient=True)
        sim.run_steps(3, {i: f[:, :3] for i, f in w.feeds.items()})     # a plain run in between
        l1 = sim.train_step(w.n_steps, w.feeds, targets)
        # the gradients sum with atomics: equal up to the order of those sums
        np.testing.assert_allclose(sim.train_param(MS.TRAIN_DECODERS, 1, gradient=True), g0, rtol=0,
                                   atol=1e-6 * np.abs(g0).max())
        assert l0 == l1
        D = sim.train_param(MS.TRAIN_DECODERS, 1)
        new = (D * 0.5).astype(np.float32)
        sim.set_train_param(MS.TRAIN_DECODERS, 1, new)
        np.testing.assert_array_equal(sim.train_param(MS.TRAIN_DECODERS, 1), new)
        assert sim.train_step(w.n_steps, w.feeds, targets) != l0
        with pytest.raises(MS.MergesimError):
            sim.train_param(MS.TRAIN_CONN_DECODERS, 0)      # connection 0 has no explicit decoders
        with pytest.raises(MS.MergesimError):
            sim.set_train_param(MS.TRAIN_BIASES, 0, np.zeros(3))


@pytest.mark.parametrize("case", ["spiking", "fused", "simplified", "graph"])
def test_models_that_cannot_train_are_refused(case):
    # the chain's ensembles have decoded-space inputs, so that fusion makes fused ensemble operators
    kw = dict(n_steps=4, minibatch=2, n_ens=2, n_neurons=20, dims=2, n_eval=40)
    # (the smoothed LIF rate is never fused: the fused case uses the exact rate curve)
    ntype = {"spiking": "lif", "fused": "lif_rate"}.get(case, "softlif_rate")
    w, targets = make_train("chain", neuron_type=ntype, **kw)
    opts = dict(TRAIN)
    if case == "fused":
        opts["fuse"] = True
    if case == "simplified":
        opts["simplify"] = True
    if case == "graph":
        opts["driver"] = M.DRIVER_GRAPH
    with M.Simulator(M.model_from_spec(w.spec), minibatch=w.minibatch, **opts) as sim:
        with pytest.raises(MS.MergesimError):
            sim.train_step(w.n_steps, w.feeds, targets)


@pytest.mark.timeout(900)
def test_classifier_full_size():
    """The 784-1024-1024-10 classifier (smoothed LIF rate) at minibatch 256
    and 50 steps, in the benchmark's launch configuration: objective, every
    gradient and the probes of the run against the oracle on all 256 rows."""
    w, targets = make_train("mlp")
    _compare(w, targets, "classifier full size")
