"""Running forward-error band of a rate-mode simulation (test helper).

A float32 simulator evaluates every current, rate, product, filter update and
sum with rounding error; near-threshold rate neurons (gains up to 1e4-1e5)
turn a tiny current error into a large rate error, and a filtered value keeps
what earlier steps moved.  BandSim steps the float64 oracle and, for every
signal, a band: how far float32 evaluation can move it, propagated first-order
through the step in the oracle's own order.  Rules (gamma = 32 * 2^-24 for
every float32 dot product or sum: the sqrt(K) growth of rounding in K-term
sums up to K = 1024, with a factor of 1 to spare):

  current    dJ = |E| dx + |g| d(input) + gamma (|bias| + |E| |x| + |g| |input|)
  rate       dr = the largest change of amplitude * r(J) over [J - dJ, J + dJ]
               + gamma |r|   (rate evaluation)
  decoded    d  = |D|^T dr + gamma |D|^T |r|
  transform  dv = |T| d(pre) + gamma |T| |pre|
  filter     dy <- a dy + b dv + gamma (a |y| + b |v|)
  sum        d(sum) = sum of the bands + gamma sum |terms|

The band of each probe, per step, plus the stated 1e-5 of the probe's peak,
bounds a float32 simulator's whole-run deviation from the float64 oracle.
Rate and ReLU neurons only (a spike decision has no first-order band)."""
import numpy as np

from oracle.neurons import rate_output
from oracle.sim import OracleSim, _obj

GAMMA = 32.0 * 2.0 ** -24


class BandSim(OracleSim):
    def __init__(self, spec, minibatch=1):
        super().__init__(spec, minibatch=minibatch, param_dtype=np.float32)
        if any(self.neuron_type[i] == "lif" for i in self.neuron_type):
            raise ValueError("error bands are defined for rate neurons only")
        self.band_data = {pi: [] for pi in range(len(spec.probes))}
        self.dy = {ci: np.zeros_like(v) for ci, v in self.y.items()}
        self.dyp = {pi: np.zeros_like(v) for pi, v in self.yp.items()}

    def band(self, probe_index):
        """Band of a probe record, [B, steps, width]."""
        return np.stack(self.band_data[probe_index], axis=1)

    def _rate(self, i, J):
        e = self.spec.ensembles[i]
        return rate_output(self.neuron_type[i], J, e.tau_rc, e.tau_ref, e.amplitude)

    def _pre(self, ci, out, dout):
        """Value read by connection ci and its band (before the transform)."""
        c = self.spec.connections[ci]
        kind, i = c.pre
        if kind == "node":
            v, dv = out[("node", i)], dout[("node", i)]
        elif kind == "neurons":
            v, dv = out[("ens", i)], dout[("ens", i)]
        else:
            D = self.conn_dec[ci]
            r, dr = out[("ens", i)], dout[("ens", i)]
            v = r @ D
            dv = dr @ np.abs(D) + GAMMA * (np.abs(r) @ np.abs(D))
        if c.pre_slice is not None:
            v, dv = v[:, c.pre_slice[0]:c.pre_slice[1]], dv[:, c.pre_slice[0]:c.pre_slice[1]]
        return v, dv

    def _value(self, ci, out, dout):
        v, dv = self._pre(ci, out, dout)
        T = self.conn_T[ci]
        if np.ndim(T) == 0:
            return v * T, abs(T) * dv + GAMMA * abs(T) * np.abs(v)
        return v @ T.T, dv @ np.abs(T).T + GAMMA * (np.abs(v) @ np.abs(T).T)

    def _step(self, feeds, k_local):
        spec, B = self.spec, self.B
        out, dout = {}, {}
        incoming = {}
        for ci, c in enumerate(spec.connections):
            incoming.setdefault(_obj(c.post), []).append(ci)

        def deliver(ci):
            c = spec.connections[ci]
            if c.synapse is not None:
                return self.y[ci], self.dy[ci]
            return self._value(ci, out, dout)

        for obj in self.order:
            kind, i = obj
            if kind == "node":
                node = spec.nodes[i]
                if node.passthrough:
                    val, dval, mag = np.zeros((B, node.size)), np.zeros((B, node.size)), np.zeros((B, node.size))
                    for ci in incoming.get(obj, []):
                        c = spec.connections[ci]
                        s0, s1 = c.post_slice or (0, node.size)
                        v, dv = deliver(ci)
                        val[:, s0:s1] += v
                        dval[:, s0:s1] += dv
                        mag[:, s0:s1] += np.abs(v)
                    dval += GAMMA * mag
                elif i in feeds:
                    val = np.asarray(feeds[i][:, k_local, :], np.float64)
                    dval = np.zeros_like(val)
                else:
                    base = np.zeros(node.size) if node.value is None else np.asarray(node.value, np.float64)
                    val = np.broadcast_to(base, (B, node.size)).copy()
                    dval = np.zeros_like(val)
                out[obj], dout[obj] = val, dval
                continue
            ens = spec.ensembles[i]
            x, dx, mx = (np.zeros((B, ens.dims)) for _ in range(3))
            nin, dn, mn = (np.zeros((B, ens.n_neurons)) for _ in range(3))
            for ci in incoming.get(obj, []):
                c = spec.connections[ci]
                post_ens = c.post[0] == "ens"
                tgt, dt_, mt = (x, dx, mx) if post_ens else (nin, dn, mn)
                s0, s1 = c.post_slice or (0, tgt.shape[1])
                v, dv = deliver(ci)
                tgt[:, s0:s1] += v
                dt_[:, s0:s1] += dv
                mt[:, s0:s1] += np.abs(v)
            dx += GAMMA * mx
            dn += GAMMA * mn
            E, g, b = self.enc[i], self.gain[i], self.bias[i]
            J = b[None, :] + x @ E.T + g[None, :] * nin
            scale = np.abs(b)[None, :] + np.abs(x) @ np.abs(E).T + np.abs(g)[None, :] * np.abs(nin)
            dJ = dx @ np.abs(E).T + np.abs(g)[None, :] * dn + GAMMA * scale
            r = self._rate(i, J)
            dr = np.maximum(np.abs(self._rate(i, J + dJ) - r), np.abs(r - self._rate(i, J - dJ))) + GAMMA * np.abs(r)
            out[obj], dout[obj] = r, dr
        for ci, c in enumerate(spec.connections):
            if c.synapse is not None:
                a, b1 = self.conn_a[ci]
                v, dv = self._value(ci, out, dout)
                self.dy[ci] = a * self.dy[ci] + b1 * dv + GAMMA * (a * np.abs(self.y[ci]) + b1 * np.abs(v))
                self.y[ci] = a * self.y[ci] + b1 * v
        for pi, p in enumerate(spec.probes):
            kind, i = p.target
            if kind == "node":
                v, dv = out[("node", i)], dout[("node", i)]
            elif kind == "neurons":
                v, dv = out[("ens", i)], dout[("ens", i)]
                if p.neuron_slice is not None:
                    v, dv = v[:, p.neuron_slice[0]:p.neuron_slice[1]], dv[:, p.neuron_slice[0]:p.neuron_slice[1]]
            else:
                D = self.dec[(i, "identity")]
                r, dr = out[("ens", i)], dout[("ens", i)]
                v, dv = r @ D, dr @ np.abs(D) + GAMMA * (np.abs(r) @ np.abs(D))
            if p.synapse is not None:
                a, b1 = self.probe_a[pi]
                self.dyp[pi] = a * self.dyp[pi] + b1 * dv + GAMMA * (a * np.abs(self.yp[pi]) + b1 * np.abs(v))
                self.yp[pi] = a * self.yp[pi] + b1 * v
                v, dv = self.yp[pi], self.dyp[pi]
            self.probe_data[pi].append(np.array(v, copy=True))
            self.band_data[pi].append(np.array(dv, copy=True))
        self.step += 1
