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
