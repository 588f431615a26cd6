"""Unmerged float64 stepper: the definition of one simulation timestep.

What a step computes (paper Sec. 2.1.3, Fig. 2: a connection is a DotInc of the
pre value into a signal reset to zero each step, then a synaptic filter, then a
copy into the post's input; Sec. 3.1: minibatch runs equal independent runs,
feeds are [batch, timesteps, dims]; Sec. 4.1.1: readers see a signal after all
writes to it).  Readings where the paper is silent:

  * step k (1-based) is time k*dt and reads feed row k-1
  * objects run in topological order of the connections that have no synapse;
    such a connection delivers T (pre value) within the same step.  A cycle of
    unfiltered connections is an error.
  * a filtered connection delivers its filter state as left by the previous
    step; after every object has run, each filter updates with this step's
    value:  y <- a y + (1 - a) v,  a = exp(-dt / tau)  (zero-order hold), where
    v = T (pre value) is the post-sized (transformed) value
  * ensemble input current J = bias + E_hat x + gain * (neuron-space input)
  * probes sample after the filter updates; a probe synapse is a lowpass on the
    probed value
  * initial state: V = 0, refractory time 0, filter states 0
  * PES learning (Sec. 5.1's pes benchmark; Fig. 7: one weight matrix per
    batch row): a connection with a learning rule decodes with its own
    decoders D^b [n, k] per batch row, initially the solved (or given)
    decoders.  Connections into ("learning", c) sum into the rule's error
    input e [B, k] (filtered ones deliver their state as left by the previous
    step, like any filtered connection).  After every object has run, and
    with the error and the activity filter read before any filter updates,
        D^b <- D^b - (kappa * dt / n) * outer(a^b, e^b)
    where a is the pre activity filter's state as left by the previous step
    (a <- p a + (1 - p) s updates after the weights are read, p =
    exp(-dt / pre_synapse)), or this step's activities s when the rule has no
    pre_synapse.  The learned connection's own filter update reads the
    decoders from before this step's change.

Every batch row is independent; parameters are shared across the batch
(learned decoders are per batch row).

``param_dtype=np.float32`` rounds every stored parameter (scaled encoders,
biases, gains, decoders, transforms, filter coefficients) to float32 before the
float64 simulation, matching what a float32 simulator stores; the arithmetic
stays float64.

Two measuring instruments for the spike disagreement a float32 simulator
cannot avoid (the defaults leave the float64 arithmetic above unchanged):
``current_dtype=np.float32`` rounds every input current J to float32 before
the neuron update and changes nothing else; ``arith_dtype=np.float32`` runs the
whole step -- state, currents, neuron update, products, filters -- in float32
(parameters rounded to float32 as with ``param_dtype``).

``direct`` lists ensembles whose neurons are replaced by the exact function of
their represented value (used by the closed-form integrator and circular
convolution pins).

Pins: tests/test_oracle_sim.py (integrator ramp in direct mode, DFT circular
convolution in direct mode, lowpass step/impulse response, LIF closed-form spike
steps through a node-driven ensemble, brute force against scalar.py, minibatch
equivalence).  Whole-network spiking trajectories: parity unpinned beyond these.
"""
from __future__ import annotations

import math
from typing import Dict, List, Optional

import numpy as np

from .build import apply_function, build_params, function_size
from .neurons import lif_step, rate_output


class CycleError(ValueError):
    pass


def _ref_size(spec, ref) -> int:
    kind, i = ref
    if kind == "node":
        return spec.nodes[i].size
    if kind == "ens":
        return spec.ensembles[i].dims
    if kind == "neurons":
        return spec.ensembles[i].n_neurons
    raise ValueError(ref)


def _obj(ref):
    """Object a reference belongs to (ensembles and their neurons are one
    object; a learning rule's error input is its own)."""
    kind, i = ref
    if kind == "learning":
        return ("learning", i)
    return ("node", i) if kind == "node" else ("ens", i)


class OracleSim:
    def __init__(self, spec, minibatch: int = 1, param_dtype=np.float64,
                 direct: frozenset = frozenset(), neuron_type: Optional[str] = None,
                 record_current: tuple = (), current_dtype=np.float64, arith_dtype=np.float64):
        self.spec = spec
        self.round_current = current_dtype == np.float32
        self.dtype = np.float32 if arith_dtype == np.float32 else np.float64
        if self.dtype == np.float32:
            param_dtype = np.float32
        self.record_current = tuple(record_current)
        self.B = int(minibatch)
        self.dt = float(spec.dt)
        self.direct = frozenset(direct)
        self.neuron_type = {i: (neuron_type or e.neuron_type)
                            for i, e in enumerate(spec.ensembles)}
        P = build_params(spec, self.direct)
        dt_ = self.dtype
        rnd = (lambda a: np.asarray(a, np.float64).astype(np.float32).astype(dt_)) \
            if param_dtype == np.float32 else (lambda a: np.asarray(a, np.float64))
        self.gain = {i: rnd(v) for i, v in P.gain.items()}
        self.bias = {i: rnd(v) for i, v in P.bias.items()}
        self.enc = {i: rnd(v) for i, v in P.scaled_encoders.items()}
        self.dec = {k: rnd(v) for k, v in P.decoders.items()}
        self.conn_dec = []
        self.conn_T = []
        self.conn_a = []
        for c in spec.connections:
            if c.pre[0] == "ens":
                self.conn_dec.append(rnd(c.decoders) if c.decoders is not None
                                     else self.dec.get((c.pre[1], c.function)))
            else:
                self.conn_dec.append(None)
            T = c.transform
            self.conn_T.append(float(rnd(T)) if np.ndim(T) == 0 else rnd(T))
            if c.synapse is not None:
                a = math.exp(-self.dt / c.synapse)
                self.conn_a.append((float(rnd(a)), float(rnd(1.0 - a))))
            else:
                self.conn_a.append(None)
        # learning rules: per learned connection (kappa dt / n, pre filter coefficients)
        self.learned = [ci for ci, c in enumerate(spec.connections) if c.learning_rule is not None]
        self.pes_coef, self.pes_a = {}, {}
        for ci in self.learned:
            c = spec.connections[ci]
            if c.pre[0] != "ens" or c.pre[1] in self.direct or c.pre_slice is not None:
                raise ValueError("a learning rule needs a decoded connection from neurons, without pre slice")
            n = spec.ensembles[c.pre[1]].n_neurons
            self.pes_coef[ci] = float(rnd(c.learning_rule.learning_rate * self.dt / n))
            tau = c.learning_rule.pre_synapse
            if tau is not None:
                a = math.exp(-self.dt / tau)
                self.pes_a[ci] = (float(rnd(a)), float(rnd(1.0 - a)))
        for ci, c in enumerate(spec.connections):
            if c.post[0] == "learning":
                if c.post[1] not in self.pes_coef:
                    raise ValueError("error connection into a connection without a learning rule")
        self.probe_a = []
        for p in spec.probes:
            if p.synapse is not None:
                a = math.exp(-self.dt / p.synapse)
                self.probe_a.append((float(rnd(a)), float(rnd(1.0 - a))))
            else:
                self.probe_a.append(None)
        self.order = self._topological_order()
        self.reset()

    # ------------------------------------------------------------------ structure
    def _topological_order(self) -> List[tuple]:
        spec = self.spec
        objs = [("node", i) for i in range(len(spec.nodes))] + \
               [("ens", i) for i in range(len(spec.ensembles))]
        succ: Dict[tuple, List[tuple]] = {o: [] for o in objs}
        indeg = {o: 0 for o in objs}
        for c in spec.connections:
            if c.synapse is None and c.post[0] != "learning":
                a, b = _obj(c.pre), _obj(c.post)
                if a == b:
                    raise CycleError("unfiltered self-connection")
                succ[a].append(b)
                indeg[b] += 1
        ready = [o for o in objs if indeg[o] == 0]
        order = []
        while ready:
            o = ready.pop(0)
            order.append(o)
            for b in succ[o]:
                indeg[b] -= 1
                if indeg[b] == 0:
                    ready.append(b)
        if len(order) != len(objs):
            raise CycleError("cycle of connections without a synapse")
        return order

    def reset(self):
        B, spec, f = self.B, self.spec, self.dtype
        self.V = {i: np.zeros((B, e.n_neurons), f) for i, e in enumerate(spec.ensembles)
                  if i not in self.direct}
        self.ref = {i: np.zeros((B, e.n_neurons), f) for i, e in enumerate(spec.ensembles)
                    if i not in self.direct}
        self.y = {ci: np.zeros((B, self._post_width(c)), f)
                  for ci, c in enumerate(spec.connections) if c.synapse is not None}
        self.yp = {pi: np.zeros((B, self._probe_width(p)), f)
                   for pi, p in enumerate(spec.probes) if p.synapse is not None}
        self.W = {ci: np.broadcast_to(self.conn_dec[ci], (B,) + self.conn_dec[ci].shape).astype(f)
                  for ci in self.learned}
        self.abar = {ci: np.zeros((B, spec.ensembles[spec.connections[ci].pre[1]].n_neurons), f)
                     for ci in self.learned if ci in self.pes_a}
        self.step = 0
        self.probe_data = {pi: [] for pi in range(len(spec.probes))}
        self.current_rec = {i: ([], []) for i in self.record_current}

    def _post_width(self, c) -> int:
        if c.post_slice is not None:
            return c.post_slice[1] - c.post_slice[0]
        if c.post[0] == "learning":
            return self.conn_dec[c.post[1]].shape[1]
        return _ref_size(self.spec, c.post)

    def _probe_width(self, p) -> int:
        if p.target[0] == "neurons" and p.neuron_slice is not None:
            return p.neuron_slice[1] - p.neuron_slice[0]
        return _ref_size(self.spec, p.target)

    # ------------------------------------------------------------------- values
    def _pre_value(self, ci, out) -> np.ndarray:
        """Value read by connection ci from its pre object this step, [B, k]."""
        c = self.spec.connections[ci]
        kind, i = c.pre
        if kind == "node":
            v = out[("node", i)]
        elif kind == "neurons":
            v = out[("ens", i)]
        else:
            if i in self.direct:
                v = apply_function(c.function, out[("ens_x", i)])
            elif ci in self.W:      # this batch row's own decoders: [B, 1, n] @ [B, n, k]
                v = np.matmul(out[("ens", i)][:, None, :], self.W[ci])[:, 0, :]
            else:
                v = out[("ens", i)] @ self.conn_dec[ci]
        if c.pre_slice is not None:
            v = v[:, c.pre_slice[0]:c.pre_slice[1]]
        return v

    def _conn_value(self, ci, out) -> np.ndarray:
        """v = T (pre value), post-sized [B, w]."""
        v = self._pre_value(ci, out)
        T = self.conn_T[ci]
        return v * T if np.ndim(T) == 0 else v @ T.T

    def _deliver(self, ci, out) -> np.ndarray:
        c = self.spec.connections[ci]
        return self.y[ci] if c.synapse is not None else self._conn_value(ci, out)

    # --------------------------------------------------------------------- step
    def _step(self, feeds: Dict[int, np.ndarray], k_local: int):
        spec, B = self.spec, self.B
        out: Dict[tuple, np.ndarray] = {}
        incoming: Dict[tuple, List[int]] = {}
        for ci, c in enumerate(spec.connections):
            incoming.setdefault(_obj(c.post), []).append(ci)
        for obj in self.order:
            kind, i = obj
            if kind == "node":
                node = spec.nodes[i]
                if node.passthrough:
                    val = np.zeros((B, node.size), self.dtype)
                    for ci in incoming.get(obj, []):
                        c = spec.connections[ci]
                        s0, s1 = c.post_slice or (0, node.size)
                        val[:, s0:s1] += self._deliver(ci, out)
                elif i in feeds:
                    val = np.asarray(feeds[i][:, k_local, :], self.dtype)
                else:
                    base = np.zeros(node.size, self.dtype) if node.value is None else \
                        np.asarray(node.value, self.dtype)
                    val = np.broadcast_to(base, (B, node.size)).copy()
                out[obj] = val
            else:
                ens = spec.ensembles[i]
                x = np.zeros((B, ens.dims), self.dtype)
                nin = np.zeros((B, ens.n_neurons), self.dtype)
                for ci in incoming.get(obj, []):
                    c = spec.connections[ci]
                    tgt = x if c.post[0] == "ens" else nin
                    s0, s1 = c.post_slice or (0, tgt.shape[1])
                    tgt[:, s0:s1] += self._deliver(ci, out)
                if i in self.direct:
                    out[("ens_x", i)] = x
                    out[obj] = None
                    continue
                J = self.bias[i][None, :] + x @ self.enc[i].T + self.gain[i][None, :] * nin
                if self.round_current:
                    J = J.astype(np.float32).astype(np.float64)
                if i in self.current_rec:
                    scale = (np.abs(self.bias[i])[None, :] + np.abs(x) @ np.abs(self.enc[i]).T
                             + np.abs(self.gain[i])[None, :] * np.abs(nin))
                    self.current_rec[i][0].append(J.copy())
                    self.current_rec[i][1].append(scale)
                if self.neuron_type[i] == "lif":
                    s, self.V[i], self.ref[i] = lif_step(J, self.V[i], self.ref[i], self.dt,
                                                         ens.tau_rc, ens.tau_ref, ens.amplitude,
                                                         dtype=self.dtype)
                else:
                    s = rate_output(self.neuron_type[i], J, ens.tau_rc, ens.tau_ref, ens.amplitude, ens.sigma)
                out[obj] = s
        # learning rules read their error input and pre activity filter
        # before any filter moves
        err, act = {}, {}
        for ci in self.learned:
            e = np.zeros((B, self.conn_dec[ci].shape[1]), self.dtype)
            for cj in incoming.get(("learning", ci), []):
                c = spec.connections[cj]
                s0, s1 = c.post_slice or (0, e.shape[1])
                e[:, s0:s1] += self._deliver(cj, out)
            err[ci] = e
            act[ci] = self.abar[ci] if ci in self.abar else out[("ens", spec.connections[ci].pre[1])]
        # filter updates run after every reader of the old filter state
        for ci, c in enumerate(spec.connections):
            if c.synapse is not None:
                a, one_minus_a = self.conn_a[ci]
                self.y[ci] = a * self.y[ci] + one_minus_a * self._conn_value(ci, out)
        # weight changes (after the learned connections' filters read the old
        # decoders), then the pre activity filters
        for ci in self.learned:
            self.W[ci] = self.W[ci] - self.pes_coef[ci] * (act[ci][:, :, None] * err[ci][:, None, :])
            if ci in self.abar:
                p_, one_minus_p = self.pes_a[ci]
                self.abar[ci] = p_ * self.abar[ci] + one_minus_p * out[("ens", spec.connections[ci].pre[1])]
        # probes sample after the updates
        for pi, p in enumerate(spec.probes):
            kind, i = p.target
            if kind == "node":
                v = out[("node", i)]
            elif kind == "neurons":
                v = out[("ens", i)]
                if p.neuron_slice is not None:
                    v = v[:, p.neuron_slice[0]:p.neuron_slice[1]]
            else:
                v = out[("ens_x", i)] if i in self.direct else out[("ens", i)] @ self.dec[(i, "identity")]
            if p.synapse is not None:
                a, one_minus_a = self.probe_a[pi]
                self.yp[pi] = a * self.yp[pi] + one_minus_a * v
                v = self.yp[pi]
            self.probe_data[pi].append(np.array(v, copy=True))
        self.step += 1

    def run_steps(self, n_steps: int, feeds: Optional[Dict[int, np.ndarray]] = None):
        """Advance n_steps; feeds map node index -> [B, n_steps, size]."""
        feeds = feeds or {}
        for i, f in feeds.items():
            f = np.asarray(f)
            assert f.shape[0] == self.B and f.shape[1] >= n_steps, (i, f.shape)
        for k in range(n_steps):
            self._step(feeds, k)

    def data(self, probe_index: int) -> np.ndarray:
        """Recorded probe values, [B, steps_since_reset, width]."""
        d = self.probe_data[probe_index]
        if not d:
            return np.zeros((self.B, 0, self._probe_width(self.spec.probes[probe_index])))
        return np.stack(d, axis=1)

    def current_data(self, ens: int):
        """Input current J of an ensemble named in record_current, and the
        magnitude of its terms |bias| + |x| |E|^T + |gain| |neuron input|, both
        [B, steps_since_reset, n_neurons].  Recording changes no arithmetic."""
        J, S = self.current_rec[ens]
        return np.stack(J, axis=1), np.stack(S, axis=1)

    # -------------------------------------------------------------------- state
    def get_state(self):
        return {"V": {i: v.copy() for i, v in self.V.items()},
                "ref": {i: v.copy() for i, v in self.ref.items()},
                "y": {i: v.copy() for i, v in self.y.items()},
                "yp": {i: v.copy() for i, v in self.yp.items()},
                "W": {i: v.copy() for i, v in self.W.items()},
                "abar": {i: v.copy() for i, v in self.abar.items()}}

    def set_state(self, state):
        for key in ("V", "ref", "y", "yp", "W", "abar"):
            cur = getattr(self, key)
            for i, v in state.get(key, {}).items():
                assert cur[i].shape == np.shape(v), (key, i)
                cur[i] = np.array(v, self.dtype, copy=True)
