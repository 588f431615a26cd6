"""Reference implementation of the paper's graph optimisations (Sec. 4.2) --
TEST INFRASTRUCTURE, written independently of the library's C++ planner so
that plans can be compared bit for bit.

  build_ir      model -> signals and operators (Sec. 2.1.3, Fig. 2), in the
                canonical order and with the canonical names the library's
                plan export uses
  simplify      y += x * 1 -> y += x ; copy of a never-changing signal -> reset
                to that constant (Sec. 4.2.4)
  dependencies  per signal: setters, then incrementers, then readers, then
                updaters (Sec. 4.1.1: reads see the result of all writes)
  merge keys    operator type, base array of each operand, DotInc weight shape
                (Sec. 4.2.1: mergeable when inputs and outputs share base arrays)
  plan_ops      greedy (n = 1) or bounded breadth-first tree search (Sec. 4.2.2):
                commit the first group of the n-step plan that schedules the
                most operators (equal counts: the plan finishing in fewer
                steps); ties: larger first group, then lower key id
  sort_metablocks   Alg. 1 (Sec. 4.2.3)
  sort_signals_ops  Alg. 2 (Sec. 4.2.3)
  lower         per-group index arrays (slices where contiguous)

Pins (tests/test_planner_ref.py): the Fig. 4 planning example (golden fixture),
brute-force shortest schedules on random small DAGs for unbounded depth,
partition / type / dependency invariants, and sorting invariants (a
permutation; disjoint read blocks become contiguous and in operator order).
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

FEED, RESET, COPY, COPY_INC, ELEM_INC, DOT_INC, LIF, LIF_RATE, LOWPASS, ENS = range(10)
BDOT_INC, PES = 11, 12          # learned decoding (per batch row) and its PES update
TYPE_NAMES = ["Feed", "Reset", "Copy", "CopyInc", "ElementwiseInc", "DotInc", "SimLIF",
              "SimLIFRate", "Lowpass", "Ensemble", "SynapseScatter", "LearnedDotInc", "PES"]
MAX_FUSED_DECODED = 16


@dataclass
class Sig:
    name: str
    rows: int
    cols: int = 1
    batched: bool = True
    base: int = -1
    value: Optional[np.ndarray] = None


@dataclass
class Ref:
    sig: int
    start: int
    length: int


@dataclass
class Op:
    type: int
    name: str
    dst: Optional[Ref] = None
    src: Optional[Ref] = None
    a: Optional[Ref] = None
    V: Optional[Ref] = None
    ref: Optional[Ref] = None
    node: int = -1
    reset_value: Optional[np.ndarray] = None
    bias: Optional[Ref] = None                 # fused ensemble: bias parameter
    decs: list = field(default_factory=list)   # fused ensemble: [(D param, d output)]
    lif: bool = True
    kind: int = 0                              # neuron type: 0 LIF, 1 LIF rate, 2 ReLU


@dataclass
class IR:
    sigs: List[Sig] = field(default_factory=list)
    ops: List[Op] = field(default_factory=list)
    bases: List[Tuple[str, bool, int]] = field(default_factory=list)   # (name, batched, cols)
    fed_rows: Dict[int, int] = field(default_factory=dict)
    probes: List[Ref] = field(default_factory=list)


def _fn_size(fn, dims):
    return 1 if fn == "product" else dims


def _fn_tag(fn):
    return "prod" if fn == "product" else "id"


# ------------------------------------------------------------------ IR build
def build_ir(spec) -> IR:
    ir = IR()
    base_ids: Dict[str, int] = {}

    def base(batched, cols):
        name = "state" if batched else ("vec" if cols == 1 else f"mat{cols}")
        if name not in base_ids:
            base_ids[name] = len(ir.bases)
            ir.bases.append((name, batched, 1 if batched else cols))
        return base_ids[name]

    def sig(name, rows, cols=1, batched=True, value=None):
        ir.sigs.append(Sig(name, rows, cols, batched, base(batched, cols), value))
        return len(ir.sigs) - 1

    def whole(s):
        return Ref(s, 0, ir.sigs[s].rows)

    def op(t, name, **kw):
        ir.ops.append(Op(t, name, **kw))
        return ir.ops[-1]

    nodes, ens, conns = spec.nodes, spec.ensembles, spec.connections

    def learn_width(ci):
        c = conns[ci]
        if c.decoders is not None:
            return np.asarray(c.decoders).shape[1]
        return _fn_size(c.function, ens[c.pre[1]].dims)

    def width(kind, i, fn="identity"):
        if kind == "learning":
            return learn_width(i)
        if kind == "node":
            return nodes[i].size
        if kind == "ens":
            return _fn_size(fn, ens[i].dims)
        return ens[i].n_neurons

    has_x = [False] * len(ens)
    has_nin = [False] * len(ens)
    fns: List[List[str]] = [[] for _ in ens]
    for c in conns:
        if c.post[0] == "ens":
            has_x[c.post[1]] = True
        if c.post[0] == "neurons":
            has_nin[c.post[1]] = True
        if c.pre[0] == "ens" and c.decoders is None and c.learning_rule is None \
                and c.function not in fns[c.pre[1]]:
            fns[c.pre[1]].append(c.function)
    for p in spec.probes:
        if p.target[0] == "ens" and "identity" not in fns[p.target[1]]:
            fns[p.target[1]].append("identity")

    node_out = []
    feed_row = 0
    for i, nd in enumerate(nodes):
        s = sig(f"n{i}.out", nd.size)
        node_out.append(s)
        if nd.passthrough:
            op(RESET, f"n{i}.reset", dst=whole(s))
        elif nd.value is not None:
            v = sig(f"n{i}.value", nd.size, 1, False, np.asarray(nd.value, float))
            op(COPY, f"n{i}.const", dst=whole(s), src=whole(v))
        else:
            ir.fed_rows[i] = feed_row
            feed_row += nd.size
            op(FEED, f"n{i}.feed", dst=whole(s), node=i)

    eJ, eS, eX, eGain, dec_sig = [], [], [], [], {}
    for e, E in enumerate(ens):
        J = sig(f"e{e}.J", E.n_neurons)
        S = sig(f"e{e}.s", E.n_neurons)
        lif = E.neuron_type == "lif"
        if lif:
            V = sig(f"e{e}.V", E.n_neurons)
            R = sig(f"e{e}.ref", E.n_neurons)
        bias = sig(f"e{e}.bias", E.n_neurons, 1, False)
        X = enc = None
        if has_x[e]:
            X = sig(f"e{e}.x", E.dims)
            enc = sig(f"e{e}.enc", E.n_neurons, E.dims, False)
        G = sig(f"e{e}.gain", E.n_neurons, 1, False) if has_nin[e] else None
        decs = []
        for fn in fns[e]:
            df = _fn_size(fn, E.dims)
            d = sig(f"e{e}.d{_fn_tag(fn)}", df)
            D = sig(f"e{e}.D{_fn_tag(fn)}", df, E.n_neurons, False)
            dec_sig[(e, fn)] = d
            decs.append((fn, d, D))
        eJ.append(J); eS.append(S); eX.append(X); eGain.append(G)
        if X is not None:
            op(RESET, f"e{e}.resetx", dst=whole(X))
        op(COPY, f"e{e}.bias", dst=whole(J), src=whole(bias))
        if X is not None:
            op(DOT_INC, f"e{e}.enc", dst=whole(J), a=whole(enc), src=whole(X))
        if lif:
            op(LIF, f"e{e}.neurons", src=whole(J), dst=whole(S), V=whole(V), ref=whole(R))
        else:
            op(LIF_RATE, f"e{e}.neurons", src=whole(J), dst=whole(S),
               kind={"relu": 2, "softlif_rate": 3}.get(E.neuron_type, 1))
        for fn, d, D in decs:
            op(RESET, f"e{e}.reset{_fn_tag(fn)}", dst=whole(d))
            op(DOT_INC, f"e{e}.dec{_fn_tag(fn)}", dst=whole(d), a=whole(D), src=whole(S))

    # error inputs of the learning rules, in connection order, before any
    # connection's own signals
    err = {ci: sig(f"c{ci}.E", learn_width(ci)) for ci, c in enumerate(conns) if c.learning_rule is not None}
    for ci, c in enumerate(conns):
        kind, i = c.pre
        if c.learning_rule is not None:
            n, k = ens[i].n_neurons, learn_width(ci)
            pre = sig(f"c{ci}.xd", k)
            W = sig(f"c{ci}.W", n * k)
            act = sig(f"c{ci}.a", n) if c.learning_rule.pre_synapse is not None else eS[i]
            op(RESET, f"c{ci}.resetd", dst=whole(pre))
            op(BDOT_INC, f"c{ci}.dec", dst=whole(pre), a=whole(W), src=whole(eS[i]))
            op(RESET, f"c{ci}.resete", dst=whole(err[ci]))
            op(PES, f"c{ci}.pes", dst=whole(W), src=whole(act), a=whole(err[ci]))
            if c.learning_rule.pre_synapse is not None:
                op(LOWPASS, f"c{ci}.presyn", dst=whole(act), src=whole(eS[i]))
        elif kind == "node":
            pre = node_out[i]
        elif kind == "neurons":
            pre = eS[i]
        elif c.decoders is not None:
            cols = np.asarray(c.decoders).shape[1]
            pre = sig(f"c{ci}.xd", cols)
            D = sig(f"c{ci}.D", cols, ens[i].n_neurons, False)
            op(RESET, f"c{ci}.resetd", dst=whole(pre))
            op(DOT_INC, f"c{ci}.dec", dst=whole(pre), a=whole(D), src=whole(eS[i]))
        else:
            pre = dec_sig[(i, c.function)]
        pre_full = ir.sigs[pre].rows
        p0, p1 = c.pre_slice if c.pre_slice is not None else (0, pre_full)
        post_full = width(c.post[0], c.post[1])
        q0, q1 = c.post_slice if c.post_slice is not None else (0, post_full)
        w, k = q1 - q0, p1 - p0
        v = sig(f"c{ci}.v", w)
        scalar = np.ndim(c.transform) == 0
        if scalar:
            t = sig(f"c{ci}.t", 1, 1, False, np.array([float(c.transform)]))
        else:
            t = sig(f"c{ci}.T", w, k, False)
        y = sig(f"c{ci}.y", w) if c.synapse is not None else None
        op(RESET, f"c{ci}.resetv", dst=whole(v))
        op(ELEM_INC if scalar else DOT_INC, f"c{ci}.transform", dst=whole(v), a=whole(t),
           src=Ref(pre, p0, k))
        if y is not None:
            op(LOWPASS, f"c{ci}.synapse", dst=whole(y), src=whole(v))
        out = y if y is not None else v
        if c.post[0] == "learning":
            op(COPY_INC, f"c{ci}.deliver", dst=Ref(err[c.post[1]], q0, w), src=whole(out))
        elif c.post[0] == "neurons":
            op(ELEM_INC, f"c{ci}.deliver", dst=Ref(eJ[c.post[1]], q0, w),
               a=Ref(eGain[c.post[1]], q0, w), src=whole(out))
        else:
            tgt = eX[c.post[1]] if c.post[0] == "ens" else node_out[c.post[1]]
            op(COPY_INC, f"c{ci}.deliver", dst=Ref(tgt, q0, w), src=whole(out))

    for pi, p in enumerate(spec.probes):
        kind, i = p.target
        if kind == "node":
            target = whole(node_out[i])
        elif kind == "ens":
            target = whole(dec_sig[(i, "identity")])
        else:
            target = whole(eS[i])
            if p.neuron_slice is not None:
                target = Ref(eS[i], p.neuron_slice[0], p.neuron_slice[1] - p.neuron_slice[0])
        if p.synapse is not None:
            y = sig(f"p{pi}.y", target.length)
            op(LOWPASS, f"p{pi}.synapse", dst=whole(y), src=target)
            ir.probes.append(whole(y))
        else:
            ir.probes.append(target)
    return ir


def simplify(ir: IR) -> None:
    for o in ir.ops:
        if o.type == ELEM_INC and o.a.length == 1:
            s = ir.sigs[o.a.sig]
            if s.value is not None and s.rows == 1 and float(s.value[0]) == 1.0 \
                    and o.src.length == o.dst.length:
                o.type, o.a = COPY_INC, None
        elif o.type == COPY and not ir.sigs[o.src.sig].batched:
            o.type, o.src = RESET, None


def fuse_ensembles(ir: IR) -> None:
    """Replace each ensemble's bias, encoder, neuron and decoder operators by one
    fused operator (an implementation choice for the GPU; the step computes the
    same values).  Ensembles whose input current has other writers (neuron-space
    connections) are left alone; decoders are fused only when their outputs
    total at most MAX_FUSED_DECODED.  Spikes are kept only if something else
    reads them."""
    by_name = {o.name: k for k, o in enumerate(ir.ops)}
    sig_by_name = {s.name: k for k, s in enumerate(ir.sigs)}
    readers = {}
    for o in ir.ops:
        own_dec = o.type == DOT_INC and o.name.startswith("e") and ".dec" in o.name
        if not own_dec:
            for r in (o.src, o.a):
                if r is not None:
                    readers[r.sig] = readers.get(r.sig, 0) + 1
    for r in ir.probes:
        readers[r.sig] = readers.get(r.sig, 0) + 1
    writers = {}
    for o in ir.ops:
        if o.dst is not None and o.type not in (LIF, LIF_RATE):
            writers[o.dst.sig] = writers.get(o.dst.sig, 0) + 1
    drop, fused = set(), {}
    e = 0
    while f"e{e}.bias" in by_name and f"e{e}.neurons" in by_name:
        p = f"e{e}"
        kb, kn = by_name[p + ".bias"], by_name[p + ".neurons"]
        ke = by_name.get(p + ".enc")
        neu = ir.ops[kn]
        # the soft LIF rate is never fused (the fused kernels compute LIF, LIF rate and ReLU)
        soft = neu.type == LIF_RATE and neu.kind == 3
        if not soft and writers.get(neu.src.sig, 0) == 1 + (ke is not None):
            dec_ops = []
            total = 0
            for tag in ("id", "prod"):
                if p + ".reset" + tag in by_name and p + ".dec" + tag in by_name:
                    dec_ops.append((by_name[p + ".reset" + tag], by_name[p + ".dec" + tag]))
                    total += ir.ops[by_name[p + ".dec" + tag]].dst.length
            dec_ops.sort(key=lambda kk: kk[1])
            fuse_dec = total <= MAX_FUSED_DECODED
            f = Op(ENS, p + ".ens", V=neu.V, ref=neu.ref, lif=neu.type == LIF, kind=neu.kind,
                   bias=Ref(sig_by_name[p + ".bias"], 0, neu.src.length))
            if ke is not None:
                f.src, f.a = ir.ops[ke].src, ir.ops[ke].a
            if fuse_dec:
                f.decs = [(ir.ops[kd].a, ir.ops[kd].dst) for _, kd in dec_ops]
            if readers.get(neu.dst.sig, 0) > 0 or not fuse_dec:
                f.dst = neu.dst
            drop |= {kb, kn} | ({ke} if ke is not None else set())
            if fuse_dec:
                drop |= {k for pair in dec_ops for k in pair}
            fused[kb] = f
        e += 1
    if not fused:
        return
    ir.ops = [fused[k] if k in fused else o for k, o in enumerate(ir.ops)
              if k in fused or k not in drop]
    used = set()
    for o in ir.ops:
        for r in (o.dst, o.src, o.a, o.V, o.ref, o.bias):
            if r is not None:
                used.add(r.sig)
        for D, d in o.decs:
            used |= {D.sig, d.sig}
    used |= {r.sig for r in ir.probes}
    remap = {}
    sigs = []
    for k, sg in enumerate(ir.sigs):
        if k in used:
            remap[k] = len(sigs)
            sigs.append(sg)
    ir.sigs = sigs
    rm = lambda r: None if r is None else Ref(remap[r.sig], r.start, r.length)
    for o in ir.ops:
        o.dst, o.src, o.a, o.V, o.ref, o.bias = map(rm, (o.dst, o.src, o.a, o.V, o.ref, o.bias))
        o.decs = [(rm(D), rm(d)) for D, d in o.decs]
    ir.probes = [rm(r) for r in ir.probes]


# ------------------------------------------------------------- dependencies
def accesses(o: Op):
    """(sets, incs, reads, updates) signal ids of an operator."""
    t = o.type
    if t in (FEED, RESET):
        return [o.dst.sig], [], [], []
    if t == COPY:
        return [o.dst.sig], [], [o.src.sig], []
    if t == COPY_INC:
        return [], [o.dst.sig], [o.src.sig], []
    if t in (ELEM_INC, DOT_INC):
        return [], [o.dst.sig], [o.a.sig, o.src.sig], []
    if t == LIF:
        return [o.dst.sig], [], [o.src.sig], [o.V.sig, o.ref.sig]
    if t == LIF_RATE:
        return [o.dst.sig], [], [o.src.sig], []
    if t == LOWPASS:
        return [], [], [o.src.sig], [o.dst.sig]
    if t == BDOT_INC:
        return [], [o.dst.sig], [o.a.sig, o.src.sig], []
    if t == PES:
        return [], [], [o.src.sig, o.a.sig], [o.dst.sig]
    if t == ENS:
        sets = ([o.dst.sig] if o.dst is not None else []) + [d.sig for _, d in o.decs]
        reads = [o.src.sig] if o.src is not None else []
        upds = [o.V.sig, o.ref.sig] if o.V is not None else []
        return sets, [], reads, upds
    raise ValueError(t)


def dependency_edges(ir: IR) -> List[Tuple[int, int]]:
    layers: Dict[int, List[List[int]]] = {}
    for k, o in enumerate(ir.ops):
        for l, sigs in enumerate(accesses(o)):
            for s in sigs:
                if not ir.sigs[s].batched:
                    continue
                L = layers.setdefault(s, [[], [], [], []])[l]
                if not L or L[-1] != k:
                    L.append(k)
    edges = []
    for s in sorted(layers):
        if len(layers[s][0]) > 1:
            raise ValueError(f"signal {ir.sigs[s].name} has more than one setter")
        prev = None
        for L in layers[s]:
            if not L:
                continue
            if prev is not None:
                edges += [(a, b) for a in prev for b in L if a != b]
            prev = L
    return edges


def merge_key(ir: IR, o: Op):
    b = lambda r: ir.sigs[r.sig].base
    t = o.type
    if t == FEED:
        return (FEED,)
    if t == RESET:
        return (RESET, b(o.dst))
    if t in (COPY, COPY_INC):
        return (t, b(o.dst), b(o.src))
    if t == ELEM_INC:
        return (t, b(o.dst), b(o.a), b(o.src))
    if t == DOT_INC:
        return (t, b(o.dst), b(o.a), b(o.src), o.a.length, o.src.length)
    if t == LIF:
        return (t, b(o.src), b(o.dst), b(o.V), b(o.ref))
    if t == LIF_RATE:
        return (t, b(o.src), b(o.dst), o.kind)
    if t == BDOT_INC:
        return (t, b(o.dst), b(o.a), b(o.src), o.dst.length, o.src.length)
    if t == PES:
        return (t, b(o.dst), b(o.src), b(o.a), o.a.length, o.src.length)
    if t == ENS:
        bb = lambda r: -1 if r is None else ir.sigs[r.sig].base
        key = (t, o.kind, bb(o.src), bb(o.a), 0 if o.src is None else o.src.length,
               bb(o.bias), bb(o.dst), bb(o.V), bb(o.ref))
        for D, d in o.decs:
            key += (bb(D), d.length, bb(d))
        return key
    return (t, b(o.dst), b(o.src))


# ------------------------------------------------------------------ planning
def plan_ops(n_ops: int, keys: Sequence[int], edges: Sequence[Tuple[int, int]],
             depth: int) -> List[List[int]]:
    """Order operators into merged groups.  keys[i] is the merge key id of op i
    (ids in first-appearance order); at each step every key's ready operators
    form one candidate group; the candidate starting the best `depth`-step plan
    (most operators scheduled) is committed.  depth=1 is the greedy planner."""
    succ = [[] for _ in range(n_ops)]
    indeg = [0] * n_ops
    for a, b in edges:
        succ[a].append(b)
        indeg[b] += 1
    # cycle check
    deg = list(indeg)
    queue = [i for i in range(n_ops) if deg[i] == 0]
    for i in queue:
        for t in succ[i]:
            deg[t] -= 1
            if deg[t] == 0:
                queue.append(t)
    if len(queue) != n_ops:
        raise ValueError("cycle")
    scheduled = [False] * n_ops

    def ready_groups(indeg_, done):
        groups: Dict[int, List[int]] = {}
        for i in range(n_ops):
            if not done[i] and indeg_[i] == 0:
                groups.setdefault(keys[i], []).append(i)
        return groups

    def schedule(indeg_, done, ops):
        indeg2, done2 = list(indeg_), list(done)
        for i in ops:
            done2[i] = True
            for t in succ[i]:
                indeg2[t] -= 1
        return indeg2, done2

    def best_value(indeg_, done, d):
        """(ops scheduled, -steps used) of the best plan of at most d steps."""
        best = None
        if d == 0:
            return (0, 0)
        for k, ops in ready_groups(indeg_, done).items():
            if d == 1:
                cand = (len(ops), -1)
            else:
                i2, d2 = schedule(indeg_, done, ops)
                rest = best_value(i2, d2, d - 1)
                cand = (len(ops) + rest[0], rest[1] - 1)
            if best is None or cand > best:
                best = cand
        return best if best is not None else (0, 0)

    plan = []
    while not all(scheduled):
        cands = ready_groups(indeg, scheduled)
        choice = None
        for k in sorted(cands):
            ops = cands[k]
            value = (len(ops), -1)
            if depth > 1:
                i2, d2 = schedule(indeg, scheduled, ops)
                rest = best_value(i2, d2, depth - 1)
                value = (len(ops) + rest[0], rest[1] - 1)
            rank = (value, len(ops))
            if choice is None or rank > choice[0]:
                choice = (rank, k)
        ops = sorted(cands[choice[1]])
        indeg, scheduled = schedule(indeg, scheduled, ops)
        plan.append(ops)
    return plan


# ------------------------------------------------------------------- sorting
def read_refs(o: Op) -> List[Ref]:
    t = o.type
    if t in (COPY, COPY_INC):
        return [o.src]
    if t in (ELEM_INC, DOT_INC):
        return [o.a, o.src]
    if t == LIF:
        return [o.src, o.V, o.ref]
    if t == LIF_RATE:
        return [o.src]
    if t == LOWPASS:
        return [o.src, o.dst]
    if t == BDOT_INC:
        return [o.a, o.src]
    if t == PES:
        return [o.src, o.a, o.dst]
    if t == ENS:
        refs = ([o.src, o.a] if o.src is not None else []) + [o.bias]
        refs += [o.V, o.ref] if o.V is not None else []
        return refs + [D for D, _ in o.decs]
    return []


@dataclass
class ReadBlock:
    group: int
    slot: int
    base: int
    size: int
    sigs: List[int]


def read_blocks(ir: IR, groups: List[List[int]]) -> List[ReadBlock]:
    blocks = []
    for gi, g in enumerate(groups):
        for slot in range(len(read_refs(ir.ops[g[0]]))):
            sigs = []
            for oi in g:
                s = read_refs(ir.ops[oi])[slot].sig
                if s not in sigs:
                    sigs.append(s)
            size = sum(ir.sigs[s].rows * ir.sigs[s].cols for s in sigs)
            blocks.append(ReadBlock(gi, slot, ir.sigs[sigs[0]].base, size, sigs))
    return blocks


def sort_metablocks(metas: List[frozenset], block_size: Dict[int, int]) -> List[int]:
    """Order meta-blocks (sets of read-block ids) so that large read blocks end
    up contiguous (Sec. 4.2.3, Alg. 1).  Meta-blocks are appended one at a
    time; the next one is the remaining meta-block that best matches the last
    one appended, by the section's four criteria in order of precedence:

      1. it contains the active read block (the block being laid out: at
         first the largest; once no remaining meta-block contains it, the
         largest block of the last meta-block takes over for later choices);
      2. it contains every read block of the last meta-block;
      3. its Hamming distance to the last meta-block is smallest;
      4. it contains the last meta-block's read blocks, the larger the better
         (compared block by block, largest first);

    then the lowest id.  Returns meta-block ids in layout order."""
    left = list(range(len(metas)))
    if not block_size:
        return left
    def size_order(blocks):
        return sorted(blocks, key=lambda bid: (-block_size[bid], bid))
    active = size_order(block_size)[0]
    # before anything is placed, a meta-block holding the active block plays
    # the part of the last one
    last = metas[next(m for m in left if active in metas[m])]
    placed = []
    while left:
        active_left = any(active in metas[m] for m in left)
        ranked_blocks = size_order(last)

        def rank(m):
            s = metas[m]
            return (active_left and active not in s,
                    not last <= s,
                    len(s ^ last),
                    tuple(bid not in s for bid in ranked_blocks),
                    m)
        best = min(left, key=rank)
        if not active_left and last:
            active = ranked_blocks[0]
        left.remove(best)
        placed.append(best)
        last = metas[best]
    return placed


def _settle(ir: IR, groups: List[List[int]], blocks: List[ReadBlock], meta_sigs: List[List[int]],
            meta_sets: List[frozenset], order: Dict[int, List[int]], passes: int) -> None:
    """Order operators and signals inside meta-blocks (Sec. 4.2.3, Alg. 2).
    For one read block b: (1) b's group takes the order in which b's signals
    lie in memory; (2) every read block c of that group has its signals
    rearranged, each meta-block within its own positions (so the meta-block
    layout of Alg. 1 stays), into the group's new operator order.  Blocks are
    taken from the smallest to the largest, so larger blocks settle last and
    win conflicts; passes repeat until one leaves everything as it was, at
    most `passes` of them."""
    pos = {s: i for base in order for i, s in enumerate(order[base])}
    visit = sorted(range(len(blocks)), key=lambda bid: (blocks[bid].size, bid))
    of_group: Dict[int, List[int]] = {}
    for bid, blk in enumerate(blocks):
        of_group.setdefault(blk.group, []).append(bid)
    metas_of = {bid: [m for m in range(len(meta_sets)) if bid in meta_sets[m]] for bid in range(len(blocks))}

    def read(op, slot):
        r = read_refs(ir.ops[op])[slot]
        return r.sig, r.start

    def ops_follow_layout(blk):
        groups[blk.group] = sorted(groups[blk.group], key=lambda op: (pos[read(op, blk.slot)[0]],
                                                                       read(op, blk.slot)[1]))

    def signals_follow_ops(bid):
        blk = blocks[bid]
        rank: Dict[int, int] = {}
        for op in groups[blk.group]:
            rank.setdefault(read(op, blk.slot)[0], len(rank))
        for m in metas_of[bid]:
            spots = sorted(pos[s] for s in meta_sigs[m])
            for spot, sig in zip(spots, sorted(meta_sigs[m], key=rank.__getitem__)):
                order[blk.base][spot] = sig
                pos[sig] = spot

    for _ in range(passes):
        before = ([list(g) for g in groups], {b: list(o) for b, o in order.items()})
        for bid in visit:
            ops_follow_layout(blocks[bid])
            for other in of_group[blocks[bid].group]:
                signals_follow_ops(other)
        if before == ([list(g) for g in groups], order):
            break


def sort_signals_ops(ir: IR, groups: List[List[int]], passes: int = 10):
    """Signal layout of every base array (meta-blocks ordered by Alg. 1, then
    operators and signals settled by Alg. 2); reorders the operators inside
    groups in place.  Meta-blocks: the signals of one base array that take
    part in exactly the same read blocks, numbered by first appearance."""
    blocks = read_blocks(ir, groups)
    member: Dict[int, List[int]] = {}
    for bi, b in enumerate(blocks):
        for s in b.sigs:
            member.setdefault(s, []).append(bi)
    meta_index: Dict[Tuple[int, Tuple[int, ...]], int] = {}
    meta_sigs: List[List[int]] = []
    meta_sets: List[frozenset] = []
    meta_base: List[int] = []
    for s, sg in enumerate(ir.sigs):
        key = (sg.base, tuple(member.get(s, [])))
        if key not in meta_index:
            meta_index[key] = len(meta_sigs)
            meta_sigs.append([])
            meta_sets.append(frozenset(member.get(s, [])))
            meta_base.append(sg.base)
        meta_sigs[meta_index[key]].append(s)
    order: Dict[int, List[int]] = {}
    for base in range(len(ir.bases)):
        ids = [m for m in range(len(meta_sigs)) if meta_base[m] == base]
        sizes = {bi: b.size for bi, b in enumerate(blocks) if b.base == base}
        local = sort_metablocks([meta_sets[m] for m in ids], sizes)
        order[base] = [s for li in local for s in meta_sigs[ids[li]]]
    _settle(ir, groups, blocks, meta_sigs, meta_sets, order, passes)
    return order


# ------------------------------------------------------------------ lowering
def _operand(base, rows):
    if all(rows[i] == rows[0] + i for i in range(len(rows))):
        return {"base": base, "start": rows[0] if rows else 0}
    return {"base": base, "idx": list(rows)}


def lower_group(ir: IR, offset: Dict[int, int], g: List[int]) -> dict:
    o0 = ir.ops[g[0]]
    t = o0.type
    row = lambda r, i: offset[r.sig] + r.start + i
    base = lambda r: ir.sigs[r.sig].base
    out = {"type": TYPE_NAMES[t], "ops": [ir.ops[i].name for i in g]}
    if t == FEED:
        d, fr = [], []
        for oi in g:
            o = ir.ops[oi]
            d += [row(o.dst, i) for i in range(o.dst.length)]
            fr += [ir.fed_rows[o.node] + i for i in range(o.dst.length)]
        out.update(rows=len(d), dst=_operand(base(o0.dst), d), feed_rows=fr)
    elif t == RESET:
        d = [row(ir.ops[oi].dst, i) for oi in g for i in range(ir.ops[oi].dst.length)]
        out.update(rows=len(d), dst=_operand(base(o0.dst), d))
    elif t == COPY:
        d, s = [], []
        for oi in g:
            o = ir.ops[oi]
            d += [row(o.dst, i) for i in range(o.dst.length)]
            s += [row(o.src, i) for i in range(o.dst.length)]
        out.update(rows=len(d), dst=_operand(base(o0.dst), d), src=_operand(base(o0.src), s))
    elif t in (COPY_INC, ELEM_INC):
        entries = []
        for oi in g:
            o = ir.ops[oi]
            for i in range(o.dst.length):
                a = row(o.a, 0 if o.a.length == 1 else i) if t == ELEM_INC else None
                entries.append((row(o.dst, i), row(o.src, i), a))
        uniq: List[int] = []
        groups_: Dict[int, List[int]] = {}
        for e, (d, _, _) in enumerate(entries):
            if d not in groups_:
                groups_[d] = []
                uniq.append(d)
            groups_[d].append(e)
        src, av, ptr = [], [], [0]
        for d in uniq:
            for e in groups_[d]:
                src.append(entries[e][1])
                av.append(entries[e][2])
            ptr.append(len(src))
        out.update(rows=len(uniq), dst=_operand(base(o0.dst), uniq), src=_operand(base(o0.src), src))
        if t == ELEM_INC:
            out["a"] = _operand(base(o0.a), av)
        if len(uniq) != len(entries):
            out["ptr"] = ptr
    elif t == DOT_INC:
        out.update(rows=len(g), M=o0.a.length, K=o0.src.length,
                   w_row=[offset[ir.ops[oi].a.sig] + ir.ops[oi].a.start for oi in g],
                   x_row=[row(ir.ops[oi].src, 0) for oi in g],
                   d_row=[row(ir.ops[oi].dst, 0) for oi in g])
    elif t in (BDOT_INC, PES):
        ops = [ir.ops[oi] for oi in g]
        out.update(rows=len(g), M=o0.dst.length if t == BDOT_INC else o0.a.length, K=o0.src.length,
                   w_row=[row(o.a if t == BDOT_INC else o.dst, 0) for o in ops],
                   x_row=[row(o.src, 0) for o in ops])
        if t == BDOT_INC:
            out["d_row"] = [row(o.dst, 0) for o in ops]
        else:
            out["e_row"] = [row(o.a, 0) for o in ops]
    elif t in (LIF, LIF_RATE):
        J, S, V, R = [], [], [], []
        for oi in g:
            o = ir.ops[oi]
            for i in range(o.src.length):
                J.append(row(o.src, i)); S.append(row(o.dst, i))
                if t == LIF:
                    V.append(row(o.V, i)); R.append(row(o.ref, i))
        out.update(rows=len(J), dst=_operand(base(o0.dst), S), src=_operand(base(o0.src), J))
        if t == LIF_RATE and o0.kind in (2, 3):
            out["neuron"] = o0.kind
        if t == LIF:
            out.update(V=_operand(base(o0.V), V), ref=_operand(base(o0.ref), R))
    elif t == ENS:
        ops = [ir.ops[oi] for oi in g]
        rr = lambda r: -1 if r is None else row(r, 0)
        bb = lambda r: -1 if r is None else ir.sigs[r.sig].base
        out.update(rows=len(g), d=0 if o0.src is None else o0.src.length, neuron=o0.kind,
                   enc_base=bb(o0.a), bias_base=bb(o0.bias), D_base=[bb(D) for D, _ in o0.decs],
                   n=[o.bias.length for o in ops], x_row=[rr(o.src) for o in ops],
                   enc_row=[-1 if o.a is None else offset[o.a.sig] for o in ops],
                   bias_row=[rr(o.bias) for o in ops], V_row=[rr(o.V) for o in ops],
                   ref_row=[rr(o.ref) for o in ops], s_row=[rr(o.dst) for o in ops],
                   df=[d.length for _, d in o0.decs],
                   D_row=[[offset[o.decs[k][0].sig] for o in ops] for k in range(len(o0.decs))],
                   d_row=[[row(o.decs[k][1], 0) for o in ops] for k in range(len(o0.decs))])
    elif t == LOWPASS:
        y, v = [], []
        for oi in g:
            o = ir.ops[oi]
            y += [row(o.dst, i) for i in range(o.dst.length)]
            v += [row(o.src, i) for i in range(o.dst.length)]
        out.update(rows=len(y), dst=_operand(base(o0.dst), y), src=_operand(base(o0.src), v))
    return out


def make_plan(spec, planner="tree", depth=3, merge=True, sort=True, do_simplify=True,
              fuse=True) -> dict:
    """The whole pipeline; returns a dict shaped like the library's JSON export
    (without parameter values)."""
    ir = build_ir(spec)
    if do_simplify:
        simplify(ir)
    if fuse:
        fuse_ensembles(ir)
    key_ids: Dict[tuple, int] = {}
    keys = []
    for k, o in enumerate(ir.ops):
        if not merge:
            keys.append(k)
            continue
        kk = merge_key(ir, o)
        if kk not in key_ids:
            key_ids[kk] = len(key_ids)
        keys.append(key_ids[kk])
    d = 1 if (planner == "greedy" or not merge) else depth
    groups = plan_ops(len(ir.ops), keys, dependency_edges(ir), d)
    if sort:
        order = sort_signals_ops(ir, groups)
    else:
        order = {b: [s for s, sg in enumerate(ir.sigs) if sg.base == b] for b in range(len(ir.bases))}
    offset = {}
    base_rows = []
    for b in range(len(ir.bases)):
        off = 0
        for s in order[b]:
            offset[s] = off
            off += ir.sigs[s].rows
        base_rows.append(off)
    probe_rows, probe_offsets = [], [0]
    for r in ir.probes:
        probe_rows += [offset[r.sig] + r.start + i for i in range(r.length)]
        probe_offsets.append(len(probe_rows))
    return {
        "bases": [{"name": n, "rows": base_rows[b], "cols": c} for b, (n, _, c) in enumerate(ir.bases)],
        "signals": [{"name": s.name, "base": s.base, "offset": offset[i], "rows": s.rows}
                    for i, s in enumerate(ir.sigs)],
        "groups": [dict(lower_group(ir, offset, g), key=keys[g[0]]) for g in groups],
        "probe_rows": probe_rows, "probe_offsets": probe_offsets,
        "feed_rows": sum(n.size for n in spec.nodes if not n.passthrough and n.value is None),
    }
