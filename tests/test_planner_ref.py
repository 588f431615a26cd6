"""Pins for oracle/planner_ref.py: the paper's planning example, brute force on
small random operator graphs, and structural invariants of plans and sorts."""
import itertools
import json
import os

import numpy as np
import pytest

from oracle import planner_ref as P
from synth import make_workload

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fig4():
    with open(os.path.join(GOLDEN, "fig4_planning.json")) as f:
        g = json.load(f)
    names = [o["name"] for o in g["ops"]]
    types = [o["type"] for o in g["ops"]]
    key_of = {}
    keys = [key_of.setdefault(t, len(key_of)) for t in types]
    edges = [(names.index(a), names.index(b)) for a, b in g["edges"]]
    return g, names, keys, edges


def test_fig4_greedy_and_tree():
    g, names, keys, edges = _fig4()
    greedy = P.plan_ops(len(names), keys, edges, depth=1)
    tree = P.plan_ops(len(names), keys, edges, depth=2)
    assert [[names[i] for i in grp] for grp in greedy] == g["expected"]["greedy"]
    assert [[names[i] for i in grp] for grp in tree] == g["expected"]["tree_depth_2"]
    # deeper searches keep the shortest plan
    assert len(P.plan_ops(len(names), keys, edges, depth=5)) == 2


def _shortest_schedule(n, keys, edges):
    """Breadth-first search over scheduled sets; a move schedules every ready
    operator of one key."""
    preds = [set() for _ in range(n)]
    for a, b in edges:
        preds[b].add(a)
    start = frozenset()
    frontier = {start}
    steps = 0
    seen = {start}
    while True:
        if any(len(s) == n for s in frontier):
            return steps
        nxt = set()
        for s in frontier:
            ready = [i for i in range(n) if i not in s and preds[i] <= s]
            for k in set(keys[i] for i in ready):
                t = s | {i for i in ready if keys[i] == k}
                if t not in seen:
                    seen.add(t)
                    nxt.add(t)
        frontier = nxt
        steps += 1


def _random_dag(rng, n, n_types):
    keys = list(rng.integers(0, n_types, n))
    # renumber keys by first appearance
    first = {}
    keys = [first.setdefault(k, len(first)) for k in keys]
    edges = [(a, b) for a in range(n) for b in range(a + 1, n) if rng.random() < 0.3]
    return keys, edges


@pytest.mark.parametrize("seed", range(40))
def test_unbounded_tree_search_is_shortest(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(3, 9))
    keys, edges = _random_dag(rng, n, int(rng.integers(2, 4)))
    plan = P.plan_ops(n, keys, edges, depth=n)
    assert len(plan) == _shortest_schedule(n, keys, edges)


@pytest.mark.parametrize("seed", range(40))
@pytest.mark.parametrize("depth", [1, 2, 3])
def test_plan_invariants(seed, depth):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(3, 12))
    keys, edges = _random_dag(rng, n, 3)
    plan = P.plan_ops(n, keys, edges, depth=depth)
    flat = [i for g in plan for i in g]
    assert sorted(flat) == list(range(n))                      # a partition
    where = {i: gi for gi, g in enumerate(plan) for i in g}
    for g in plan:
        assert len({keys[i] for i in g}) == 1                  # one operator type/key
    for a, b in edges:
        assert where[a] < where[b]                             # dependencies respected
    # greedy never beats the deeper search by more than the search allows
    if depth > 1:
        assert len(plan) <= len(P.plan_ops(n, keys, edges, depth=1)) + n


def test_metablock_sort_disjoint_blocks_is_permutation():
    metas = [frozenset({0}), frozenset({1}), frozenset({2}), frozenset()]
    sizes = {0: 5, 1: 50, 2: 7}
    out = P.sort_metablocks(metas, sizes)
    assert sorted(out) == [0, 1, 2, 3]
    assert out[0] == 1                                         # largest block first


def test_metablock_sort_keeps_largest_block_contiguous():
    # block 0 (large) spans meta-blocks {0}, {0,1}; block 1 spans {0,1}, {1}
    metas = [frozenset({1}), frozenset({0, 1}), frozenset({0}), frozenset({2})]
    sizes = {0: 100, 1: 10, 2: 1}
    out = P.sort_metablocks(metas, sizes)
    pos = {m: i for i, m in enumerate(out)}
    with0 = sorted(pos[m] for m in range(4) if 0 in metas[m])
    assert with0 == list(range(with0[0], with0[0] + len(with0)))


@pytest.mark.parametrize("name,kw", [("c2", dict(n_steps=2, minibatch=1)),
                                     ("c4", dict(n_ens=8, n_steps=2, minibatch=1))])
def test_sorted_plans_read_more_contiguously(name, kw):
    """Alg. 1/2 output is a layout in which groups read contiguous slices at
    least as often as in build order (sorting never makes a plan worse here)."""
    w = make_workload(name, **kw)
    def idx_operands(plan):
        n = 0
        for g in plan["groups"]:
            for k in ("src", "a", "V", "ref"):
                if k in g and "idx" in g[k]:
                    n += 1
        return n
    sorted_plan = P.make_plan(w.spec, sort=True)
    unsorted_plan = P.make_plan(w.spec, sort=False)
    assert idx_operands(sorted_plan) <= idx_operands(unsorted_plan)
    # layouts are permutations: every signal placed once, no overlap
    for plan in (sorted_plan, unsorted_plan):
        for b, base in enumerate(plan["bases"]):
            spans = sorted((s["offset"], s["offset"] + s["rows"]) for s in plan["signals"] if s["base"] == b)
            assert spans[0][0] == 0 and spans[-1][1] == base["rows"]
            assert all(x[1] == y[0] for x, y in zip(spans, spans[1:]))


# --------------------------------------------------------------------- sorting
# Abstract sorting instances: one state base array, signals of given sizes,
# groups of operators that read one signal per slot (Copy: one slot; Lowpass:
# two, its input and its own state).  Only the reads matter to the sort.

def _instance(rows, group_reads):
    ir = P.IR()
    ir.bases = [("state", True, 1)]
    for k, r in enumerate(rows):
        ir.sigs.append(P.Sig(name=f"s{k}", rows=r, base=0))
    groups = []
    for g in group_reads:
        ids = []
        for reads in g:
            ref = [P.Ref(s, 0, rows[s]) for s in reads]
            if len(reads) == 1:
                o = P.Op(type=P.COPY, name=f"o{len(ir.ops)}", src=ref[0], dst=ref[0])
            else:
                o = P.Op(type=P.LOWPASS, name=f"o{len(ir.ops)}", src=ref[0], dst=ref[1])
            ir.ops.append(o)
            ids.append(len(ir.ops) - 1)
        groups.append(ids)
    return ir, groups


def _blocks(ir, groups):
    """Read blocks: per group and slot, the signals in operator order."""
    out = []
    for g in groups:
        for slot in range(len(P.read_refs(ir.ops[g[0]]))):
            seq = []
            for op in g:
                s = P.read_refs(ir.ops[op])[slot].sig
                if s not in seq:
                    seq.append(s)
            out.append(seq)
    return out


def _in_order(ir, seq, order):
    """The block's signals lie back to back, in the operators' order."""
    off, o = {}, 0
    for s in order:
        off[s] = o
        o += ir.sigs[s].rows
    return all(off[b] == off[a] + ir.sigs[a].rows for a, b in zip(seq, seq[1:]))


def _contiguous(seq, order):
    pos = sorted(order.index(s) for s in seq)
    return pos == list(range(pos[0], pos[0] + len(pos)))


def _score(ir, groups, order):
    """Elements read as contiguous in-order slices (the reads the sort is for)."""
    return sum(sum(ir.sigs[s].rows for s in b) for b in _blocks(ir, groups) if _in_order(ir, b, order))


@pytest.mark.parametrize("seed", range(30))
def test_disjoint_read_blocks_become_contiguous_and_in_order(seed):
    """When no signal is read by two groups or slots, every read block is one
    meta-block, and Alg. 1 then Alg. 2 must make every block a contiguous
    slice in its operators' order -- whatever the initial layout and operator
    order (random here), and for two-slot groups too (Alg. 2 step 2 puts the
    second slot's signals in the order step 1 gave the operators)."""
    rng = np.random.default_rng(500 + seed)
    n_groups = int(rng.integers(2, 5))
    slots = [int(rng.integers(1, 3)) for _ in range(n_groups)]
    n_ops = [int(rng.integers(2, 5)) for _ in range(n_groups)]
    n_sig = sum(s * k for s, k in zip(slots, n_ops)) + int(rng.integers(0, 3))   # some unread
    sigs = list(rng.permutation(n_sig))
    rows = [int(r) for r in rng.integers(1, 5, n_sig)]
    reads = []
    for s, k in zip(slots, n_ops):
        reads.append([tuple(sigs.pop() for _ in range(s)) for _ in range(k)])
    ir, groups = _instance(rows, reads)
    order = P.sort_signals_ops(ir, groups)[0]
    assert sorted(order) == list(range(n_sig))
    for seq in _blocks(ir, groups):
        assert _in_order(ir, seq, order), (seq, order)


def test_overlap_hand_worked():
    """The situation Sec. 4.2.3 describes: one group reads two blocks, b (the
    inputs v) and c (the states y).  Layout after Alg. 1 (larger block c
    first, canonical order inside meta-blocks): y0 y1 y2 | v2 v0 v1.  Alg. 2
    visits b first (smaller): step 1 orders the operators by b, (2, 0, 1),
    which breaks c; step 2 rearranges c to y2 y0 y1.  Visiting c then changes
    nothing, and a second pass confirms it.  Without step 2 the visit of c
    would reorder the operators to (0, 1, 2) and break b."""
    #          y0 y1 y2 v2 v0 v1
    rows = [2, 2, 2, 1, 1, 1]
    v = {2: 3, 0: 4, 1: 5}
    ir, groups = _instance(rows, [[(v[k], k) for k in range(3)]])
    order = P.sort_signals_ops(ir, groups)[0]
    assert order == [2, 0, 1, 3, 4, 5]
    assert groups == [[2, 0, 1]]
    for seq in _blocks(ir, groups):
        assert _in_order(ir, seq, order)


def test_larger_block_wins_a_conflict():
    """Two two-slot groups over seven signals whose reads conflict (signals 0
    and 4 are read by both groups, paired differently), so no layout serves
    every block.  Blocks (signals in operator order, elements): group 0 slot 0
    [4, 1, 6] 6, slot 1 [6, 5, 0] 5; group 1 slot 0 [4, 3] 4, slot 1 [0, 4] 3.
    Alg. 2 visits blocks smallest first, so the largest block (group 0 slot 0)
    has the last word and ends as a contiguous slice in its operators' order
    (Sec. 4.2.3: later sorting only breaks the orderings of earlier, smaller
    blocks); visiting them largest first leaves no block in order here."""
    rows = [1, 3, 1, 2, 2, 3, 1]
    ir, groups = _instance(rows, [[(4, 6), (1, 5), (6, 0)], [(4, 0), (3, 4)]])
    order = P.sort_signals_ops(ir, groups)[0]
    blocks = _blocks(ir, groups)
    sizes = [sum(rows[s] for s in b) for b in blocks]
    assert sizes == [6, 5, 4, 3]
    assert _in_order(ir, blocks[0], order)


def _random_small_instance(rng):
    n = int(rng.integers(3, 7))
    rows = [int(r) for r in rng.integers(1, 5, n)]
    reads = []
    for _ in range(int(rng.integers(2, 4))):
        nslot = int(rng.integers(1, 3))
        reads.append([tuple(int(s) for s in rng.integers(0, n, nslot)) for _ in range(int(rng.integers(2, 4)))])
    return _instance(rows, reads)


def test_sort_against_brute_force_on_tiny_instances():
    """Up to six signals, two or three groups of two or three operators with
    overlapping reads: every signal order and every operator order per group
    is tried.  The heuristic is not optimal (Sec. 4.2.3 says no efficient
    optimal method is known), so this states its measured quality as bounds:
    the largest read block is always contiguous (it is Alg. 1's first active
    block), the elements read as contiguous in-order slices are at least 0.2
    of the optimum on every instance and 0.8 of it on average (measured: worst
    0.36, mean 0.89 over these 40 instances); Alg. 1's contiguity alone
    reaches at least 0.3 of the best order of signals on every instance, 0.8 on
    average (measured: worst 0.56, mean 0.92)."""
    rng = np.random.default_rng(77)
    ratios, ratios1 = [], []
    for _ in range(40):
        ir, groups = _random_small_instance(rng)
        n = len(ir.sigs)
        blocks0 = _blocks(ir, groups)
        g2 = [list(g) for g in groups]
        order = P.sort_signals_ops(ir, g2)[0]
        sizes = [sum(ir.sigs[s].rows for s in b) for b in blocks0]
        largest = max(range(len(blocks0)), key=lambda i: (sizes[i], -i))
        assert _contiguous(blocks0[largest], order)
        best = 0
        best1 = 0
        for perm in itertools.permutations(range(n)):
            perm = list(perm)
            best1 = max(best1, sum(sz for b, sz in zip(blocks0, sizes) if _contiguous(b, perm)))
            for ops in itertools.product(*[itertools.permutations(g) for g in groups]):
                best = max(best, _score(ir, [list(o) for o in ops], perm))
        got = _score(ir, g2, order)
        got1 = sum(sz for b, sz in zip(blocks0, sizes) if _contiguous(b, order))
        ratios.append(got / best if best else 1.0)
        ratios1.append(got1 / best1 if best1 else 1.0)
    print(f"in-order score / optimum: worst {min(ratios):.2f}, mean {np.mean(ratios):.2f}; "
          f"Alg. 1 contiguity / optimum: worst {min(ratios1):.2f}, mean {np.mean(ratios1):.2f}")
    assert min(ratios) >= 0.2 and np.mean(ratios) >= 0.8
    assert min(ratios1) >= 0.3 and np.mean(ratios1) >= 0.8


def test_metablock_criteria_hand_worked():
    """Alg. 1's criteria one at a time.  Blocks 0, 1, 2 of sizes 10, 5, 3;
    meta-blocks A {0}, B {0, 1}, C {0, 2}, D {1}, E {2}.  Block 0 is active
    first and A (the first meta-block holding it) stands for the last one:
    A itself matches best (Hamming distance 0); then B and C both hold block
    0 and all of A, at distance 1 from A, and both hold A's block 0: the lower
    id, B.  C is the last one holding block 0.  From C = {0, 2} no remaining
    meta-block holds block 0 or contains C; E {2} is at distance 1, D {1} at
    3: E, then D."""
    metas = [frozenset({0}), frozenset({0, 1}), frozenset({0, 2}), frozenset({1}), frozenset({2})]
    out = P.sort_metablocks(metas, {0: 10, 1: 5, 2: 3})
    assert out == [0, 1, 2, 4, 3]


def test_metablock_criterion_two_keeps_supersets_together():
    """Criterion 2 before 3: after A {0, 1}, both X {0, 1, 2, 3} and Y {0} hold
    the active block 0; X contains all of A (Hamming distance 2), Y does not
    (distance 1).  Containment ranks first: A, X, Y (Hamming alone would give
    A, Y, X)."""
    metas = [frozenset({0, 1}), frozenset({0, 1, 2, 3}), frozenset({0})]
    assert P.sort_metablocks(metas, {0: 10, 1: 5, 2: 2, 3: 2}) == [0, 1, 2]


def test_metablock_criterion_four_prefers_the_larger_block():
    """Criterion 4 compares the last meta-block's blocks largest first.  After
    A {0, 1, 2} (active block 0, size 20, held by no other), Y {2, 9} (id 1)
    and X {1, 9} (id 2) tie on criteria 1-3 (neither contains A, both at
    distance 3).  X holds block 1 (size 6), Y block 2 (size 5): A, X, Y (the
    lower id, or comparing the smaller blocks first, would pick Y)."""
    metas = [frozenset({0, 1, 2}), frozenset({2, 9}), frozenset({1, 9})]
    assert P.sort_metablocks(metas, {0: 20, 1: 6, 2: 5, 9: 1}) == [0, 2, 1]


def test_signal_sort_needs_a_second_pass():
    """Why Alg. 2 makes several passes (Sec. 4.2.3).  Group S copies q0, q1;
    group L reads (p_k, q_(2-k)), k = 0..2 (all signals one element).  Alg. 1
    lays out p0 p1 p2 | q2 | q0 q1.  Pass 1 visits S's block (2 elements)
    first, which is in order; then L's blocks (3 each): L's order by p is
    (p0, p1, p2), so step 2 rearranges q0 q1 into L's order, q1 q0 -- which
    breaks S.  Pass 2 re-sorts S's operators to (q1, q0); pass 3 changes
    nothing.  Final: p0 p1 p2 q2 q1 q0, every block in order; a single pass
    leaves S out of order."""
    ir, groups = _instance([1] * 6, [[(3,), (4,)], [(0, 5), (1, 4), (2, 3)]])
    order = P.sort_signals_ops(ir, groups)[0]
    assert order == [0, 1, 2, 5, 4, 3]
    assert groups == [[1, 0], [2, 3, 4]]
    assert all(_in_order(ir, b, order) for b in _blocks(ir, groups))
