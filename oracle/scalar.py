"""Pure-Python (no numpy in the stepping) per-object, per-neuron interpreter.

It restates the step of sim.py element by element with ``math`` scalars and
explicit loops -- a second, independently written reading of the same step
definition -- so that tiny models can brute-force-check the vectorised stepper.
It reuses only the build step's parameters (gain, bias, decoders), which are
pinned separately.  Slow: use a handful of neurons and steps.
"""
import math


def _lif_scalar(J, V, ref, dt, tau_rc, tau_ref, amp):
    integ = dt - ref
    if integ < 0.0:
        integ = 0.0
    if integ > dt:
        integ = dt
    V = V - (J - V) * math.expm1(-integ / tau_rc)
    ref = ref - dt
    if ref < 0.0:
        ref = 0.0
    if V > 1.0:
        since = 0.0
        if J > 1.0:
            q = (V - 1.0) / (J - 1.0)
            since = integ if q >= 1.0 else min(-tau_rc * math.log1p(-q), integ)
        return amp / dt, 0.0, tau_ref - since
    return 0.0, (V if V > 0.0 else 0.0), ref


def _rate_scalar(J, tau_rc, tau_ref, amp):
    if J <= 1.0:
        return 0.0
    return amp / (tau_ref + tau_rc * math.log1p(1.0 / (J - 1.0)))


def _sizes(spec, ref):
    k, i = ref
    if k == "node":
        return spec.nodes[i].size
    if k == "ens":
        return spec.ensembles[i].dims
    return spec.ensembles[i].n_neurons


def run_scalar(spec, params, n_steps, feeds=None, minibatch=1, neuron_type=None):
    """Simulate and return {probe index: nested lists [B][T][w]}."""
    feeds = feeds or {}
    dt = spec.dt
    nn = len(spec.nodes)
    # object ids: nodes 0..nn-1, ensembles nn..
    def oid(ref):
        return ref[1] if ref[0] == "node" else nn + ref[1]
    n_obj = nn + len(spec.ensembles)
    # depth-first topological order over unfiltered connections
    deps = [[] for _ in range(n_obj)]
    for c in spec.connections:
        if c.synapse is None:
            deps[oid(c.post)].append(oid(c.pre))
    order, mark = [], [0] * n_obj

    def visit(o):
        if mark[o] == 2:
            return
        if mark[o] == 1:
            raise ValueError("cycle without synapse")
        mark[o] = 1
        for p in deps[o]:
            visit(p)
        mark[o] = 2
        order.append(o)
    for o in range(n_obj):
        visit(o)

    ntype = [neuron_type or e.neuron_type for e in spec.ensembles]
    results = {}
    for b in range(minibatch):
        V = [[0.0] * e.n_neurons for e in spec.ensembles]
        R = [[0.0] * e.n_neurons for e in spec.ensembles]
        Y = {}
        for ci, c in enumerate(spec.connections):
            if c.synapse is not None:
                w = (c.post_slice[1] - c.post_slice[0]) if c.post_slice else _sizes(spec, c.post)
                Y[ci] = [0.0] * w
        YP = {pi: None for pi, p in enumerate(spec.probes) if p.synapse is not None}
        rec = {pi: [] for pi in range(len(spec.probes))}
        for k in range(n_steps):
            outv = [None] * n_obj   # node outputs / ensemble spikes
            def pre_value(ci):
                c = spec.connections[ci]
                kind, i = c.pre
                if kind == "node":
                    v = outv[i]
                elif kind == "neurons":
                    v = outv[nn + i]
                else:
                    D = c.decoders if c.decoders is not None else params.decoders[(i, c.function)]
                    s = outv[nn + i]
                    v = [sum(s[n] * float(D[n][j]) for n in range(len(s)))
                         for j in range(len(D[0]))]
                if c.pre_slice:
                    v = v[c.pre_slice[0]:c.pre_slice[1]]
                return v

            def conn_value(ci):
                c = spec.connections[ci]
                v = pre_value(ci)
                T = c.transform
                if not hasattr(T, "shape") or len(getattr(T, "shape", ())) == 0:
                    return [float(T) * a for a in v]
                return [sum(float(T[r][q]) * v[q] for q in range(len(v)))
                        for r in range(len(T))]

            def delivered(ci):
                return list(Y[ci]) if ci in Y else conn_value(ci)

            for o in order:
                if o < nn:
                    node = spec.nodes[o]
                    if node.passthrough:
                        val = [0.0] * node.size
                        for ci, c in enumerate(spec.connections):
                            if c.post == ("node", o):
                                s0 = c.post_slice[0] if c.post_slice else 0
                                for j, a in enumerate(delivered(ci)):
                                    val[s0 + j] += a
                    elif o in feeds:
                        val = [float(a) for a in feeds[o][b][k]]
                    else:
                        val = [0.0] * node.size if node.value is None else \
                            [float(a) for a in node.value]
                    outv[o] = val
                else:
                    ei = o - nn
                    e = spec.ensembles[ei]
                    x = [0.0] * e.dims
                    nin = [0.0] * e.n_neurons
                    for ci, c in enumerate(spec.connections):
                        if c.post[1] == ei and c.post[0] in ("ens", "neurons"):
                            tgt = x if c.post[0] == "ens" else nin
                            s0 = c.post_slice[0] if c.post_slice else 0
                            for j, a in enumerate(delivered(ci)):
                                tgt[s0 + j] += a
                    g, bi = params.gain[ei], params.bias[ei]
                    spikes = []
                    for n in range(e.n_neurons):
                        J = float(bi[n]) + float(g[n]) * nin[n]
                        for d in range(e.dims):
                            J += float(g[n]) * float(e.encoders[n][d]) * x[d]
                        if ntype[ei] == "lif":
                            s, V[ei][n], R[ei][n] = _lif_scalar(J, V[ei][n], R[ei][n], dt,
                                                                e.tau_rc, e.tau_ref, e.amplitude)
                        else:
                            s = _rate_scalar(J, e.tau_rc, e.tau_ref, e.amplitude)
                        spikes.append(s)
                    outv[o] = spikes
            for ci, c in enumerate(spec.connections):
                if ci in Y:
                    a = math.exp(-dt / c.synapse)
                    v = conn_value(ci)
                    Y[ci] = [a * yo + (1.0 - a) * vn for yo, vn in zip(Y[ci], v)]
            for pi, p in enumerate(spec.probes):
                kind, i = p.target
                if kind == "node":
                    v = list(outv[i])
                elif kind == "neurons":
                    v = list(outv[nn + i])
                    if p.neuron_slice:
                        v = v[p.neuron_slice[0]:p.neuron_slice[1]]
                else:
                    D = params.decoders[(i, "identity")]
                    s = outv[nn + i]
                    v = [sum(s[n] * float(D[n][j]) for n in range(len(s)))
                         for j in range(len(D[0]))]
                if p.synapse is not None:
                    a = math.exp(-dt / p.synapse)
                    YP[pi] = [(1.0 - a) * vn for vn in v] if YP[pi] is None else \
                        [a * yo + (1.0 - a) * vn for yo, vn in zip(YP[pi], v)]
                    v = list(YP[pi])
                rec[pi].append(v)
        for pi in rec:
            results.setdefault(pi, []).append(rec[pi])
    return results
