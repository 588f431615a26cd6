"""Training objective and its gradient through the unrolled simulation -- TEST
INFRASTRUCTURE ONLY (imported by tests/, the smoke check and the benchmark's
CPU baseline; the GPU library never calls it).

Paper Sec. 3.2: a model is trained by minimising an objective defined on probe
outputs with a gradient-descent optimiser, the gradient running back through
every step of the unrolled simulation; non-differentiable spiking neurons are
trained in their rate form.  Readings where the paper leaves details open:

  * rate neurons only (LIF rate, smoothed LIF rate, ReLU).  The spiking LIF
    step has no useful derivative; swapping it for a rate form automatically
    is not part of this library, so a model is built with rate neurons to be
    trained.  The exact LIF rate curve's slope grows without bound at
    threshold, which makes its gradients sensitive to the rounding of
    near-threshold currents; the smoothed curve (neurons.soft_lif_rate)
    bounds it;
  * every training run starts from the initial state (filter states zero);
  * objective: for each probe given a target [B, T, w], the mean over batch
    rows, steps and probe dimensions of the squared difference (the mean
    squared error); the objective is the sum over the probes given targets;
  * trained parameters: each ensemble's gain-scaled encoders E_hat [n, d] and
    biases [n]; each (ensemble, function)'s decoders [n, d_f], shared by every
    connection and probe that decodes that function; each connection's
    explicit decoders [n, k]; each connection's transform ([w, k], or a
    scalar).  Gains of neuron-space inputs, node constants and filter
    coefficients stay fixed;
  * the derivative of the LIF rate curve at J <= 1 is 0 (the curve is 0
    there); ReLU's derivative at J <= 0 is 0;
  * an optimiser step is plain gradient descent, p <- p - lr * dL/dp.

The forward pass restates OracleSim's step (sim.py: same object order, same
filter and probe timing) for rate neurons with torch float64 tensors; the
gradient is torch's reverse-mode differentiation of that forward pass (a
library primitive standing for the chain rule through the unrolled steps).

Pins (tests/test_oracle_train.py): the forward pass equals OracleSim's probe
data; every gradient equals central finite differences of the objective
computed by OracleSim (numpy, no autograd); a one-neuron, one-step model and a
filtered scalar connection against gradients worked out by hand.
"""
from __future__ import annotations

from typing import Dict, Optional

import numpy as np
import torch

from .sim import OracleSim

_FN = {"identity": 0, "product": 1}


def trainable_params(ref: OracleSim) -> Dict[tuple, np.ndarray]:
    """The trained parameters of a model, as float64 copies of the values an
    OracleSim holds (param_dtype=np.float32 gives the float32-rounded values a
    float32 simulator starts from).  Keys:
      ("enc", e)       [n, d]  gain-scaled encoders
      ("bias", e)      [n]
      ("dec", e, fn)   [n, d_f] decoders of function fn (0 identity, 1 product)
      ("cdec", c)      [n, k]  explicit decoders of connection c
      ("T", c)         [w, k] transform of connection c, or [1] for a scalar"""
    spec, P = ref.spec, {}
    for e, ens in enumerate(spec.ensembles):
        if ens.neuron_type not in ("lif_rate", "softlif_rate", "relu"):
            raise ValueError(f"ensemble {e} has neuron type {ens.neuron_type!r}: train rate neurons")
        if e in ref.enc and any(c.post == ("ens", e) for c in spec.connections):
            P[("enc", e)] = np.array(ref.enc[e], np.float64)
        P[("bias", e)] = np.array(ref.bias[e], np.float64)
    for (e, fn), D in ref.dec.items():
        used = any(c.pre == ("ens", e) and c.decoders is None and c.function == fn
                   for c in spec.connections) or \
            (fn == "identity" and any(p.target == ("ens", e) for p in spec.probes))
        if used:
            P[("dec", e, _FN[fn])] = np.array(D, np.float64)
    for ci, c in enumerate(spec.connections):
        if c.learning_rule is not None:
            raise ValueError("online learning rules are not trained by gradient descent here")
        if c.pre[0] == "ens" and c.decoders is not None:
            P[("cdec", ci)] = np.array(ref.conn_dec[ci], np.float64)
        T = ref.conn_T[ci]
        P[("T", ci)] = np.array([T], np.float64) if np.ndim(T) == 0 else np.array(T, np.float64)
    return P


def _rate(ntype, J, ens):
    """amplitude * r(J): LIF rate 1/(tau_ref + tau_rc log(1 + 1/(J - 1))) above
    J = 1, the smoothed LIF rate with rho = sigma log(1 + exp((J - 1)/sigma))
    in place of J - 1 (neurons.soft_lif_rate), ReLU max(J, 0).  The exact
    curve's J <= 1 branch is masked so that its derivative is exactly 0."""
    if ntype == "relu":   # torch.relu's derivative at J = 0 is 0 (clamp's would be 1)
        return ens.amplitude * torch.relu(J)
    if ntype == "softlif_rate":   # evaluated as in neurons.soft_lif_rate
        x = (J - 1.0) / ens.sigma
        far = x < -30.0
        xs = torch.where(far, torch.zeros_like(x), x)
        q_near = torch.log1p(1.0 / (ens.sigma * torch.logaddexp(xs, torch.zeros_like(xs))))
        xf = torch.where(far, x, torch.full_like(x, -30.0))
        q_far = torch.log1p(ens.sigma * torch.exp(xf)) - (np.log(ens.sigma) + xf)
        q = torch.where(far, q_far, q_near)
        return ens.amplitude / (ens.tau_ref + ens.tau_rc * q)
    on = J > 1.0
    Js = torch.where(on, J, torch.full_like(J, 2.0))
    r = 1.0 / (ens.tau_ref + ens.tau_rc * torch.log1p(1.0 / (Js - 1.0)))
    return ens.amplitude * torch.where(on, r, torch.zeros_like(J))


class TrainOracle:
    """Objective, gradients and gradient-descent steps of a rate-neuron model.

    ``params`` starts as trainable_params(OracleSim(spec, param_dtype=...)) and
    is updated in place by sgd(); the fixed values (gains, filter
    coefficients, node constants) come from the same OracleSim.

    ``arith=torch.float32`` runs the same forward and backward passes in
    float32 and stores the parameters in float32 after each update (a
    measuring instrument: how far float32 arithmetic alone moves the
    objective, the gradients and the trained parameters); the default is
    float64.  ``chunk=k`` sums every matrix product over its inner index in
    consecutive slices of k, one slice after the other (in float32 another,
    equally valid, rounding of the same sums: the order in which a GPU
    product kernel that walks the inner index in slices accumulates)."""

    def __init__(self, spec, minibatch: int = 1, param_dtype=np.float32, arith=torch.float64,
                 chunk: int = 0):
        self.spec = spec
        self.B = int(minibatch)
        self.tdtype = arith
        self.chunk = int(chunk)
        self.ref = OracleSim(spec, minibatch=minibatch, param_dtype=param_dtype)
        self.params = trainable_params(self.ref)
        self.order = self.ref.order

    # ------------------------------------------------------------- forward
    def _forward(self, P, n_steps, feeds):
        spec, ref, B = self.spec, self.ref, self.B
        fdt = self.tdtype
        fixed_gain = {i: torch.as_tensor(g, dtype=fdt) for i, g in ref.gain.items()}
        incoming = {}
        for ci, c in enumerate(spec.connections):
            key = ("node", c.post[1]) if c.post[0] == "node" else ("ens", c.post[1])
            incoming.setdefault(key, []).append(ci)
        y = {ci: torch.zeros(B, ref._post_width(c), dtype=fdt)
             for ci, c in enumerate(spec.connections) if c.synapse is not None}
        yp = {pi: torch.zeros(B, ref._probe_width(p), dtype=fdt)
              for pi, p in enumerate(spec.probes) if p.synapse is not None}
        rec = {pi: [] for pi in range(len(spec.probes))}

        def mm(a, b):
            if not self.chunk or a.shape[1] <= self.chunk:
                return a @ b
            acc = a[:, :self.chunk] @ b[:self.chunk]
            for k0 in range(self.chunk, a.shape[1], self.chunk):
                acc = acc + a[:, k0:k0 + self.chunk] @ b[k0:k0 + self.chunk]
            return acc

        def dec_of(ci):
            c = spec.connections[ci]
            if c.decoders is not None:
                return P[("cdec", ci)]
            return P[("dec", c.pre[1], _FN[c.function])]

        def conn_value(ci, out):
            c = spec.connections[ci]
            kind, i = c.pre
            if kind == "node":
                v = out[("node", i)]
            elif kind == "neurons":
                v = out[("ens", i)]
            else:
                v = mm(out[("ens", i)], dec_of(ci))
            if c.pre_slice is not None:
                v = v[:, c.pre_slice[0]:c.pre_slice[1]]
            T = P[("T", ci)]
            return v * T[0] if np.ndim(spec.connections[ci].transform) == 0 else mm(v, T.T)

        def deliver(ci, out):
            return y[ci] if spec.connections[ci].synapse is not None else conn_value(ci, out)

        def summed(width, cis, out, neurons=None):
            acc = torch.zeros(B, width, dtype=fdt)
            for ci in cis:
                c = spec.connections[ci]
                if neurons is not None and (c.post[0] == "neurons") != neurons:
                    continue
                s0, s1 = c.post_slice or (0, width)
                idx = torch.arange(s0, s1)
                acc = acc.index_add(1, idx, deliver(ci, out))
            return acc

        for k in range(n_steps):
            out = {}
            for obj in self.order:
                kind, i = obj
                if kind == "node":
                    node = spec.nodes[i]
                    if node.passthrough:
                        out[obj] = summed(node.size, incoming.get(obj, []), out)
                    elif i in feeds:
                        out[obj] = torch.as_tensor(np.asarray(feeds[i][:, k, :], np.float64), dtype=fdt)
                    else:
                        base = np.zeros(node.size) if node.value is None else np.asarray(node.value, np.float64)
                        out[obj] = torch.as_tensor(np.broadcast_to(base, (B, node.size)).copy(), dtype=fdt)
                else:
                    ens = spec.ensembles[i]
                    cis = incoming.get(obj, [])
                    J = P[("bias", i)][None, :].expand(B, -1)
                    if ("enc", i) in P:
                        J = J + mm(summed(ens.dims, cis, out, neurons=False), P[("enc", i)].T)
                    if any(spec.connections[ci].post[0] == "neurons" for ci in cis):
                        J = J + fixed_gain[i][None, :] * summed(ens.n_neurons, cis, out, neurons=True)
                    out[obj] = _rate(ens.neuron_type, J, ens)
            for ci, c in enumerate(spec.connections):
                if c.synapse is not None:
                    a, one_minus_a = ref.conn_a[ci]
                    y[ci] = a * y[ci] + one_minus_a * conn_value(ci, out)
            for pi, p in enumerate(spec.probes):
                kind, i = p.target
                if kind == "node":
                    v = out[("node", i)]
                elif kind == "neurons":
                    v = out[("ens", i)]
                    if p.neuron_slice is not None:
                        v = v[:, p.neuron_slice[0]:p.neuron_slice[1]]
                else:
                    v = mm(out[("ens", i)], P[("dec", i, 0)])
                if p.synapse is not None:
                    a, one_minus_a = ref.probe_a[pi]
                    yp[pi] = a * yp[pi] + one_minus_a * v
                    v = yp[pi]
                rec[pi].append(v)
        return {pi: torch.stack(v, dim=1) if v else torch.zeros(B, 0, 0, dtype=fdt)
                for pi, v in rec.items()}

    # ------------------------------------------------------------ objective
    def loss_and_grads(self, n_steps: int, feeds: Dict[int, np.ndarray], targets: Dict[int, np.ndarray]):
        """(objective, {param key: dL/dp}, {probe: [B, T, w] data}) of one run
        from the initial state with the current parameters."""
        leaves = {k: torch.tensor(v, dtype=self.tdtype, requires_grad=True) for k, v in self.params.items()}
        probes = self._forward(leaves, n_steps, feeds)
        loss = torch.zeros((), dtype=self.tdtype)
        for pi, tgt in targets.items():
            t = torch.as_tensor(np.asarray(tgt, np.float64)[:, :n_steps], dtype=self.tdtype)
            loss = loss + torch.mean((probes[pi] - t) ** 2)
        keys = list(leaves)
        grads = torch.autograd.grad(loss, [leaves[k] for k in keys], allow_unused=True)
        g = {k: (np.zeros_like(self.params[k]) if gk is None else gk.detach().double().numpy().copy())
             for k, gk in zip(keys, grads)}
        return float(loss.detach()), g, {pi: v.detach().double().numpy() for pi, v in probes.items()}

    def sgd(self, grads: Dict[tuple, np.ndarray], learning_rate: float):
        for k, gk in grads.items():
            p = self.params[k] - learning_rate * gk
            self.params[k] = p.astype(np.float32).astype(np.float64) if self.tdtype == torch.float32 else p


def objective_numpy(spec, minibatch, n_steps, feeds, targets, params, param_dtype=np.float32) -> float:
    """The same objective computed by OracleSim (numpy float64, no automatic
    differentiation) with the given trained parameters: the independent side
    of the finite-difference pins."""
    sim = OracleSim(spec, minibatch=minibatch, param_dtype=param_dtype)
    inv = {v: k for k, v in _FN.items()}
    for key, val in params.items():
        if key[0] == "enc":
            sim.enc[key[1]] = np.array(val, np.float64)
        elif key[0] == "bias":
            sim.bias[key[1]] = np.array(val, np.float64)
        elif key[0] == "dec":
            sim.dec[(key[1], inv[key[2]])][...] = val   # shared with the connections decoding it
        elif key[0] == "cdec":
            sim.conn_dec[key[1]] = np.array(val, np.float64)
        elif key[0] == "T":
            T = spec.connections[key[1]].transform
            sim.conn_T[key[1]] = float(val[0]) if np.ndim(T) == 0 else np.array(val, np.float64)
    sim.run_steps(n_steps, {i: f[:, :n_steps] for i, f in feeds.items()})
    loss = 0.0
    for pi, tgt in targets.items():
        loss += float(np.mean((sim.data(pi) - np.asarray(tgt, np.float64)[:, :n_steps]) ** 2))
    return loss
