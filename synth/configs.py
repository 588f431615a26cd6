"""Seeded generators for the five benchmark-shaped workloads.

Seed of workload c<k> is k.  Every object draws from its own sub-stream
``numpy.random.default_rng([seed, object_index])`` so that shrinking one part
of a model (fewer ensembles, fewer batch rows) leaves the other objects'
parameters unchanged.

  c1  integrator   1 ensemble x 100 LIF, 1-D, recurrent (paper Sec. 5.1 "integrator")
  c2  cconv        128 product ensembles x 100 LIF (2-D), D=64 real-DFT transforms
                   (paper Sec. 5.1 "cconv")
  c3  spiking MLP  784 -> 1024 LIF -> 1024 LIF -> 10 (paper Sec. 5.2.1 shape)
  c4  wide array   200 ensembles x 500 LIF x 16-D in a chain
  c5  sparse graph 5000 ensembles x 500 LIF x 16-D, fan-out 4, 32-D input
  bg  basal-ganglia-shaped: five arrays of D one-dimensional ensembles (striatum
      D1 and D2, STN, GPi, GPe) with one-to-one and all-to-all array transforms
      (paper Sec. 5.1 "basal_ganglia"; used for the planner ablation)
  pes online learning: a D-dimensional ensemble whose output weights learn the
      identity by PES, 10 batch rows (paper Sec. 5.1 "pes", Fig. 7)

All values are synthetic; no dataset is read or reproduced.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np

from .spec import PES, Connection, Ensemble, ModelSpec, Node, Probe, Workload

CONFIG_NAMES = ("c1", "c2", "c3", "c4", "c5", "bg", "pes")


def _rng(seed: int, index: int) -> np.random.Generator:
    return np.random.default_rng([seed, index])


def unit_sphere(rng, n: int, d: int) -> np.ndarray:
    """n points uniform on the unit sphere in R^d (for d == 1: +-1)."""
    if d == 1:
        return rng.choice([-1.0, 1.0], size=(n, 1))
    x = rng.standard_normal((n, d))
    return x / np.linalg.norm(x, axis=1, keepdims=True)


def unit_ball(rng, n: int, d: int, radius: float = 1.0) -> np.ndarray:
    """n points uniform in the ball of the given radius in R^d."""
    if d == 1:
        return rng.uniform(-radius, radius, size=(n, 1))
    direction = unit_sphere(rng, n, d)
    r = radius * rng.uniform(0.0, 1.0, size=(n, 1)) ** (1.0 / d)
    return direction * r


def random_orthogonal(rng, d: int) -> np.ndarray:
    """Haar-distributed orthogonal matrix (QR of a Gaussian, signs fixed)."""
    q, r = np.linalg.qr(rng.standard_normal((d, d)))
    return q * np.sign(np.diag(r))[None, :]


def lif_ensemble(rng, n: int, d: int, n_eval: int, neuron_type: str,
                 amplitude: float = 1.0) -> Ensemble:
    return Ensemble(
        n_neurons=n, dims=d,
        encoders=unit_sphere(rng, n, d),
        eval_points=unit_ball(rng, n_eval, d),
        max_rates=rng.uniform(200.0, 400.0, size=n),
        intercepts=rng.uniform(-1.0, 1.0, size=n),
        neuron_type=neuron_type, amplitude=amplitude)


# ----------------------------------------------------------------------------- c1
def make_c1(neuron_type="lif", n_steps=1000, minibatch=1, n_neurons=100) -> Workload:
    seed = 1
    m = ModelSpec(dt=0.001)
    inp = m.add_node(Node(size=1))
    e = m.add_ensemble(lif_ensemble(_rng(seed, 1), n_neurons, 1, 50, neuron_type))
    tau = 0.1
    m.connect(Connection(pre=inp, post=("ens", e), transform=tau, synapse=tau))
    m.connect(Connection(pre=("ens", e), post=("ens", e), transform=1.0, synapse=tau))
    m.probe(Probe(target=("ens", e), synapse=0.01))
    m.probe(Probe(target=("neurons", e)))
    t = np.arange(1, n_steps + 1) * m.dt
    feed = np.broadcast_to((0.5 * np.sin(2 * np.pi * t))[None, :, None],
                           (minibatch, n_steps, 1)).astype(np.float32)
    return Workload("c1", m, minibatch, n_steps, {0: np.ascontiguousarray(feed)},
                    notes="integrator: input 0.5 sin(2 pi t), recurrent lowpass 0.1")


# ----------------------------------------------------------------------------- c2
def cconv_transforms(D: int, s: float = 0.5):
    """Real-DFT factorisation of circular convolution into scalar products.

    Returns (T_A, T_B, T_out, n_products): ensemble j receives
    x = (s * alpha_j . a, s * beta_j . b) and decodes x0 * x1; the output is
    T_out @ products.  With exact products, T_out @ p == a (*) b.
    """
    assert D % 2 == 0
    n = np.arange(D)
    cos = lambda k: np.cos(2 * np.pi * k * n / D)
    msin = lambda k: -np.sin(2 * np.pi * k * n / D)
    alphas, betas, outs = [], [], []
    # DC and Nyquist coefficients are real: one product each
    for k, sign in ((0, np.ones(D)), (D // 2, (-1.0) ** n)):
        alphas.append(cos(k)); betas.append(cos(k)); outs.append(sign / D)
    for k in range(1, D // 2):
        c, si = np.cos(2 * np.pi * k * n / D), np.sin(2 * np.pi * k * n / D)
        # Re C_k = ReA ReB - ImA ImB ; Im C_k = ReA ImB + ImA ReB
        # c_n += (2/D) (Re C_k cos - Im C_k sin)
        alphas += [cos(k), msin(k), cos(k), msin(k)]
        betas += [cos(k), msin(k), msin(k), cos(k)]
        outs += [2 * c / D, -2 * c / D, -2 * si / D, -2 * si / D]
    n_prod = len(alphas)                 # 2 + 4 (D/2 - 1) = 2D - 2
    n_ens = 2 * D                        # padded with zero-input ensembles
    T_A = np.zeros((2 * n_ens, D)); T_B = np.zeros((2 * n_ens, D))
    T_out = np.zeros((D, n_ens))
    for j in range(n_prod):
        T_A[2 * j] = s * alphas[j]
        T_B[2 * j + 1] = s * betas[j]
        T_out[:, j] = outs[j] / (s * s)
    return T_A, T_B, T_out, n_ens


def make_c2(neuron_type="lif", n_steps=1000, minibatch=64, D=64, n_neurons=100,
            n_eval=1000, spike_probe_ensembles=(0, 1)) -> Workload:
    seed = 2
    m = ModelSpec(dt=0.001)
    T_A, T_B, T_out, n_ens = cconv_transforms(D)
    a = m.add_node(Node(size=D))
    b = m.add_node(Node(size=D))
    p_in = m.add_node(Node(size=2 * n_ens, passthrough=True))
    p_out = m.add_node(Node(size=n_ens, passthrough=True))
    out = m.add_node(Node(size=D, passthrough=True))
    syn = 0.005
    m.connect(Connection(pre=a, post=p_in, transform=T_A, synapse=syn))
    m.connect(Connection(pre=b, post=p_in, transform=T_B, synapse=syn))
    for j in range(n_ens):
        rng = _rng(seed, 10 + j)
        e = m.add_ensemble(Ensemble(
            n_neurons=n_neurons, dims=2, encoders=unit_sphere(rng, n_neurons, 2),
            eval_points=unit_ball(rng, n_eval, 2),
            max_rates=rng.uniform(200, 400, n_neurons),
            intercepts=rng.uniform(-1, 1, n_neurons), neuron_type=neuron_type))
        m.connect(Connection(pre=p_in, post=("ens", e), transform=1.0,
                             pre_slice=(2 * j, 2 * j + 2)))
        m.connect(Connection(pre=("ens", e), post=p_out, transform=1.0,
                             function="product", post_slice=(j, j + 1)))
    m.connect(Connection(pre=p_out, post=out, transform=T_out, synapse=syn))
    m.probe(Probe(target=out))
    for j in spike_probe_ensembles:
        m.probe(Probe(target=("neurons", j)))
    feeds = {}
    for node_idx, sub in ((0, 1), (1, 2)):
        rng = _rng(seed, sub)
        v = rng.standard_normal((minibatch, D))
        v /= np.linalg.norm(v, axis=1, keepdims=True)
        feeds[node_idx] = np.ascontiguousarray(
            np.broadcast_to(v[:, None, :], (minibatch, n_steps, D))).astype(np.float32)
    return Workload("c2", m, minibatch, n_steps, feeds,
                    notes="circular-convolution shaped: 128 product ensembles, DFT transforms")


# ----------------------------------------------------------------------------- c3
def make_c3(neuron_type="lif", n_steps=50, minibatch=256, n_in=784, n_hidden=1024,
            n_out=10, amplitude=0.01) -> Workload:
    seed = 3
    m = ModelSpec(dt=0.001)
    inp = m.add_node(Node(size=n_in))
    readout = m.add_node(Node(size=n_out, passthrough=True))
    layers = []
    for li in range(2):
        rng = _rng(seed, 1 + li)
        e = m.add_ensemble(Ensemble(
            n_neurons=n_hidden, dims=1, encoders=np.ones((n_hidden, 1)),
            eval_points=np.zeros((1, 1)),
            max_rates=rng.uniform(200, 400, n_hidden),
            intercepts=rng.uniform(-1, 1, n_hidden),
            neuron_type=neuron_type, amplitude=amplitude))
        layers.append(e)

    def glorot(rng, fan_out, fan_in):
        return rng.standard_normal((fan_out, fan_in)) * np.sqrt(2.0 / (fan_in + fan_out))

    W1 = glorot(_rng(seed, 11), n_hidden, n_in)
    W2 = glorot(_rng(seed, 12), n_hidden, n_hidden)
    W3 = glorot(_rng(seed, 13), n_out, n_hidden)
    m.connect(Connection(pre=inp, post=("neurons", layers[0]), transform=W1, synapse=None))
    m.connect(Connection(pre=("neurons", layers[0]), post=("neurons", layers[1]),
                         transform=W2, synapse=0.005))
    m.connect(Connection(pre=("neurons", layers[1]), post=readout, transform=W3,
                         synapse=0.005))
    m.probe(Probe(target=readout))
    m.probe(Probe(target=("neurons", layers[0])))
    m.probe(Probe(target=("neurons", layers[1])))
    rng = _rng(seed, 20)
    img = rng.uniform(0.0, 1.0, size=(minibatch, n_in))
    feed = np.ascontiguousarray(
        np.broadcast_to(img[:, None, :], (minibatch, n_steps, n_in))).astype(np.float32)
    return Workload("c3", m, minibatch, n_steps, {0: feed},
                    notes="spiking MLP 784-1024-1024-10, Glorot-normal weights, U[0,1] input")


# ----------------------------------------------------------------------------- c4
def make_c4(neuron_type="lif", n_steps=500, minibatch=512, n_ens=200, n_neurons=500,
            dims=16, n_eval=1000, spike_probe_ensembles=(0, None)) -> Workload:
    seed = 4
    m = ModelSpec(dt=0.001)
    inp = m.add_node(Node(size=dims))
    syn = 0.005
    ens = []
    for i in range(n_ens):
        ens.append(m.add_ensemble(lif_ensemble(_rng(seed, 100 + i), n_neurons, dims,
                                               n_eval, neuron_type)))
    m.connect(Connection(pre=inp, post=("ens", ens[0]), transform=1.0, synapse=syn))
    for i in range(n_ens - 1):
        T = random_orthogonal(_rng(seed, 100000 + i), dims)
        m.connect(Connection(pre=("ens", ens[i]), post=("ens", ens[i + 1]), transform=T,
                             synapse=syn))
    m.probe(Probe(target=("ens", ens[-1]), synapse=syn))
    for j in spike_probe_ensembles:
        m.probe(Probe(target=("neurons", ens[-1] if j is None else ens[j])))
    rng = _rng(seed, 1)
    v = unit_ball(rng, minibatch, dims, radius=0.5)
    feed = np.ascontiguousarray(
        np.broadcast_to(v[:, None, :], (minibatch, n_steps, dims))).astype(np.float32)
    return Workload("c4", m, minibatch, n_steps, {0: feed},
                    notes="wide ensemble array: chain of 16-D ensembles, orthogonal transforms")


# ----------------------------------------------------------------------------- c5
def make_c5(neuron_type="lif", n_steps=1000, minibatch=1, n_ens=5000, n_neurons=500,
            dims=16, n_eval=1000, fan_out=4, n_input_targets=100, in_dims=32,
            n_probed=16) -> Workload:
    seed = 5
    m = ModelSpec(dt=0.001)
    inp = m.add_node(Node(size=in_dims))
    syn = 0.005
    for i in range(n_ens):
        m.add_ensemble(lif_ensemble(_rng(seed, 100 + i), n_neurons, dims, n_eval,
                                    neuron_type))
    wiring = _rng(seed, 2)
    for i in range(n_ens):
        others = wiring.choice(n_ens - 1, size=min(fan_out, n_ens - 1), replace=False)
        others = np.where(others >= i, others + 1, others)   # skip self
        for k, j in enumerate(others):
            T = 0.5 * random_orthogonal(_rng(seed, 10_000_000 + i * fan_out + k), dims)
            m.connect(Connection(pre=("ens", i), post=("ens", int(j)), transform=T,
                                 synapse=syn))
    tgt = _rng(seed, 3).choice(n_ens, size=min(n_input_targets, n_ens), replace=False)
    for k, j in enumerate(tgt):
        T = _rng(seed, 20_000_000 + k).standard_normal((dims, in_dims)) / np.sqrt(in_dims)
        m.connect(Connection(pre=inp, post=("ens", int(j)), transform=T, synapse=syn))
    probed = _rng(seed, 4).choice(n_ens, size=min(n_probed, n_ens), replace=False)
    for j in probed:
        m.probe(Probe(target=("ens", int(j)), synapse=syn))
    m.probe(Probe(target=("neurons", int(probed[0]))))
    feed = _rng(seed, 1).uniform(-1.0, 1.0, size=(minibatch, n_steps, in_dims))
    return Workload("c5", m, minibatch, n_steps, {0: feed.astype(np.float32)},
                    notes="sparse random graph of 16-D ensembles, fan-out 4, 32-D input")


# ----------------------------------------------------------------------------- bg
def make_bg(neuron_type="lif", n_steps=1000, minibatch=1, D=64, n_neurons=50, n_eval=300) -> Workload:
    """Basal-ganglia-shaped network (the paper names the benchmark without its
    structure; this follows the usual action-selection circuit).  Five arrays
    of D one-dimensional ensembles, each with an input and an output
    passthrough of width D: striatum D1 (input weight 1.2), striatum D2 (0.8)
    and STN (1.0) read the D utilities; D1 -> GPi and D2 -> GPe inhibit one to
    one (-1, lowpass 0.008); STN excites GPi and GPe all to all (0.9, lowpass
    0.002); GPe inhibits GPi and STN one to one (-0.3, lowpass 0.008), which
    closes the STN-GPe loop.  Neurons have positive encoders and intercepts
    U[0.2, 0.9], so each ensemble responds only above a threshold.  The GPi
    output is probed (lowpass 0.01) with the spikes of one GPi ensemble.
    Feed: seeded utilities U[0, 1]^D per batch row, constant in time."""
    seed = 6
    m = ModelSpec(dt=0.001)
    u = m.add_node(Node(size=D))
    eye, ones = np.eye(D), np.ones((D, D))

    def array(k):
        inp = m.add_node(Node(size=D, passthrough=True))
        out = m.add_node(Node(size=D, passthrough=True))
        ens = []
        for j in range(D):
            rng = _rng(seed, 1000 * k + j)
            e = m.add_ensemble(Ensemble(
                n_neurons=n_neurons, dims=1, encoders=np.ones((n_neurons, 1)),
                eval_points=rng.uniform(0.0, 1.2, size=(n_eval, 1)),
                max_rates=rng.uniform(200.0, 400.0, n_neurons),
                intercepts=rng.uniform(0.2, 0.9, n_neurons), neuron_type=neuron_type))
            m.connect(Connection(pre=inp, post=("ens", e), transform=1.0, pre_slice=(j, j + 1)))
            m.connect(Connection(pre=("ens", e), post=out, transform=1.0, post_slice=(j, j + 1)))
            ens.append(e)
        return inp, out, ens

    d1_in, d1_out, _ = array(1)
    d2_in, d2_out, _ = array(2)
    stn_in, stn_out, _ = array(3)
    gpi_in, gpi_out, gpi = array(4)
    gpe_in, gpe_out, _ = array(5)
    ampa, gaba = 0.002, 0.008
    m.connect(Connection(pre=u, post=d1_in, transform=1.2 * eye, synapse=ampa))
    m.connect(Connection(pre=u, post=d2_in, transform=0.8 * eye, synapse=ampa))
    m.connect(Connection(pre=u, post=stn_in, transform=1.0 * eye, synapse=ampa))
    m.connect(Connection(pre=d1_out, post=gpi_in, transform=-1.0 * eye, synapse=gaba))
    m.connect(Connection(pre=d2_out, post=gpe_in, transform=-1.0 * eye, synapse=gaba))
    m.connect(Connection(pre=stn_out, post=gpi_in, transform=0.9 * ones, synapse=ampa))
    m.connect(Connection(pre=stn_out, post=gpe_in, transform=0.9 * ones, synapse=ampa))
    m.connect(Connection(pre=gpe_out, post=gpi_in, transform=-0.3 * eye, synapse=gaba))
    m.connect(Connection(pre=gpe_out, post=stn_in, transform=-0.3 * eye, synapse=gaba))
    m.probe(Probe(target=gpi_out, synapse=0.01))
    m.probe(Probe(target=("neurons", gpi[0])))
    rng = _rng(seed, 1)
    v = rng.uniform(0.0, 1.0, size=(minibatch, D))
    feeds = {u[1]: np.ascontiguousarray(np.broadcast_to(v[:, None, :], (minibatch, n_steps, D))).astype(np.float32)}
    return Workload("bg", m, minibatch, n_steps, feeds,
                    notes="basal-ganglia shaped: 5 arrays of D 1-D ensembles, one-to-one and all-to-all")


# ---------------------------------------------------------------------------- pes
def make_pes(neuron_type="lif", n_steps=1000, minibatch=10, D=192, neurons_per_dim=50,
             learning_rate=1e-4, pre_synapse=0.005, n_eval=100) -> Workload:
    """Online-learning benchmark shape (paper Sec. 5.1 "pes": an ensemble whose
    output weights learn by PES; Figs. 6 and 7 vary D over 64, 128, 192 and
    batch 10 inputs).  A D-dimensional input node drives an ensemble of
    neurons_per_dim * D neurons (lowpass 0.005).  The ensemble reaches a
    passthrough output node through a connection with zero initial decoders
    that learns by PES (learning rate 1e-4, pre activities lowpass 0.005;
    lowpass 0.005 on the connection); its error is output minus input (two
    connections into the rule, lowpass 0.005 each).  Probed: the output node
    (lowpass 0.01).  Feed: per batch row and dimension 0.5 sin(2 pi f t +
    phase), f ~ U[1, 5] Hz, phase ~ U[0, 2 pi)."""
    seed = 7
    m = ModelSpec(dt=0.001)
    n = neurons_per_dim * D
    inp = m.add_node(Node(size=D))
    out = m.add_node(Node(size=D, passthrough=True))
    e = m.add_ensemble(lif_ensemble(_rng(seed, 100), n, D, n_eval, neuron_type))
    syn = 0.005
    m.connect(Connection(pre=inp, post=("ens", e), transform=1.0, synapse=syn))
    c = m.connect(Connection(pre=("ens", e), post=out, decoders=np.zeros((n, D)), synapse=syn,
                             learning_rule=PES(learning_rate=learning_rate, pre_synapse=pre_synapse)))
    m.connect(Connection(pre=out, post=("learning", c), transform=1.0, synapse=syn))
    m.connect(Connection(pre=inp, post=("learning", c), transform=-1.0, synapse=syn))
    m.probe(Probe(target=out, synapse=0.01))
    rng = _rng(seed, 1)
    f = rng.uniform(1.0, 5.0, size=(minibatch, 1, D))
    ph = rng.uniform(0.0, 2 * np.pi, size=(minibatch, 1, D))
    t = (np.arange(1, n_steps + 1) * m.dt)[None, :, None]
    feed = 0.5 * np.sin(2 * np.pi * f * t + ph)
    return Workload("pes", m, minibatch, n_steps, {inp[1]: feed.astype(np.float32)},
                    notes="PES learning of the identity, zero initial decoders, per-batch-row weights")


# ------------------------------------------------------------------------ training
def make_train(kind="mlp", neuron_type="softlif_rate", seed=7, **overrides):
    """A rate-neuron model to train by gradient descent (paper Sec. 3.2) and
    seeded targets for some of its probes: (Workload, {probe: [B, T, w]}).

    Rate neurons: the smoothed LIF rate by default (the differentiable
    stand-in of a spiking LIF model; smoothing sigma 0.02 from Ensemble).

    kind "mlp": the spiking-classifier shape (784-1024-1024-10, filtered
      hidden connections, 50 steps, minibatch 256) with rate neurons of one
      maximum rate (100 Hz) and intercept (0), the usual set-up of a
      classifier to be trained (every neuron gets the same moderate gain);
      each batch row's target on the readout probe is a one-hot class vector
      drawn from the seed, at every step.
    kind "chain": the ensemble-array shape (a chain of d-dimensional
      ensembles with orthogonal transforms and lowpass synapses); targets on
      the filtered decoded output: the input vector rotated by a seeded
      orthogonal matrix, at every step.
    kind "cconv": the circular-convolution shape (product ensembles, DFT
      transforms, decoded product function, slices); targets on the output
      node: seeded values of magnitude 0.1."""
    if kind == "mlp":
        w = make_c3(neuron_type=neuron_type, **overrides)
        for e in w.spec.ensembles:
            e.max_rates = np.full(e.n_neurons, 100.0)
            e.intercepts = np.zeros(e.n_neurons)
        rng = _rng(seed, 1)
        n_out = w.spec.nodes[1].size
        cls = rng.integers(0, n_out, size=w.minibatch)
        tgt = np.zeros((w.minibatch, w.n_steps, n_out), np.float32)
        tgt[np.arange(w.minibatch), :, cls] = 1.0
        return w, {0: tgt}
    if kind == "chain":
        w = make_c4(neuron_type=neuron_type, **overrides)
        d = w.spec.nodes[0].size
        R = random_orthogonal(_rng(seed, 2), d)
        tgt = np.einsum("btd,ed->bte", w.feeds[0].astype(np.float64), R).astype(np.float32)
        return w, {0: tgt}
    if kind == "cconv":
        w = make_c2(neuron_type=neuron_type, **overrides)
        D = w.spec.nodes[4].size
        tgt = (0.1 * _rng(seed, 3).standard_normal((w.minibatch, 1, D))).astype(np.float32)
        return w, {0: np.ascontiguousarray(np.broadcast_to(tgt, (w.minibatch, w.n_steps, D)))}
    raise ValueError(f"unknown training workload {kind!r}")


_MAKERS = {"c1": make_c1, "c2": make_c2, "c3": make_c3, "c4": make_c4, "c5": make_c5, "bg": make_bg,
           "pes": make_pes}


def make_workload(name: str, **overrides) -> Workload:
    """Build workload ``name`` ("c1".."c5", "bg", "pes"); keyword overrides shrink it for tests
    (n_steps, minibatch, n_ens, n_neurons, neuron_type, ...)."""
    return _MAKERS[name](**overrides)
