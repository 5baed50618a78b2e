"""Evidence ordering (CPU).

The oracle model of the knowledge tree (oracle.ordering.TreeModel and the
orders defined on it) is pinned first: the paper's Fig. 2 example, the
fallback to retrieval order, the recency window, hand-worked staleness and
recency cases, greedy = exhaustive whenever no visited node has two cached
children still to place (Sec. 3.3), and the k! search against an independent
formulation over the cached orders. The library's C++ tree (cw_tree_*) is then
compared with the oracle on random histories: orders, depths and the greedy
walk's probe counts must be identical for every strategy.
"""
import itertools
import os

import numpy as np
import pytest

from oracle import ordering as O
from paper_2606_19667_amd import cw
from paper_2606_19667_amd import workload as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _fig2():
    d = {}
    with open(os.path.join(GOLDEN, "fig2_trie_example.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            k, v = line.split(":", 1)
            d[k.strip()] = v.split()
    return d


def _cached_orders(m: O.TreeModel):
    return [list(o) for t, o in m.served if t > m.clock - m.window]


def _single_branch(m: O.TreeModel, docs) -> bool:
    """Every node the walk can reach has at most one cached child still to place."""
    stack = [((), set(docs))]
    while stack:
        path, rest = stack.pop()
        kids = [d for d in rest if m.is_cached(path + (d,))]
        if len(kids) > 1:
            return False
        stack += [(path + (d,), rest - {d}) for d in kids]
    return True


# ---------------------------------------------------------------------------
# Oracle pins
# ---------------------------------------------------------------------------
def test_oracle_fig2_example():
    ex = _fig2()
    m = O.TreeModel(window=8)
    m.insert(ex["cached_path"])
    order, depth, probes = O.greedy_order(ex["candidates"], m.is_cached)
    assert order == ex["expected_order"] and depth == int(ex["expected_depth"][0])
    k = len(ex["candidates"])
    assert probes <= k * (k + 1) // 2
    assert O.exhaustive_order(ex["candidates"], m.is_cached) == (ex["expected_order"], depth)


def test_oracle_fallback_is_retrieval_order():
    m = O.TreeModel(window=4)
    assert O.greedy_order([5, 3, 9], m.is_cached) == ([5, 3, 9], 0, 3)     # empty tree
    m.insert([1, 2, 3])
    assert O.greedy_order([7, 8, 2], m.is_cached)[:2] == ([7, 8, 2], 0)   # no cached child of the root


def test_oracle_recency_window_expires_paths():
    m = O.TreeModel(window=3)
    m.insert([1, 2])
    for n in range(3):
        m.insert([10 + n])
    assert O.greedy_order([2, 1], m.is_cached)[1] == 0      # served 4 insertions ago
    m.insert([1, 2])
    assert O.greedy_order([2, 1], m.is_cached) == ([1, 2], 2, 3)


def test_oracle_stale_marks_hand_example():
    m = O.TreeModel(window=8)
    m.insert([1, 4])
    m.insert([1, 2, 3])
    assert O.greedy_order([1, 2, 3, 4], m.is_cached)[:2] == ([1, 2, 3, 4], 3)
    # the engine reused only document 1 of [1, 2, 3]: nodes (1, 2) and (1, 2, 3) go stale
    m.mark_stale([1, 2, 3], 1)
    assert m.is_cached((1,)) and not m.is_cached((1, 2)) and not m.is_cached((1, 2, 3))
    assert m.is_cached((1, 4))                               # a sibling branch is untouched
    assert O.greedy_order([1, 2, 3, 4], m.is_cached)[:2] == ([1, 4, 2, 3], 2)
    m.insert([1, 2, 3])                                      # served again: fresh
    assert O.greedy_order([1, 2, 3, 4], m.is_cached)[:2] == ([1, 2, 3, 4], 3)
    m.mark_stale([1, 2, 3], 0)                               # nothing reused: the whole path
    assert not m.is_cached((1,)) and O.greedy_order([1, 2, 3, 4], m.is_cached)[1] == 0


def test_oracle_baseline_orders_hand_examples():
    assert O.retrieval_order([3, 1, 2]) == [3, 1, 2]
    assert O.sorted_order([30, 1, 200]) == [1, 30, 200]
    m = O.TreeModel(window=3)
    m.insert([5, 6])
    m.insert([7])
    # 7 served last, then 6 and 5 (same time: retrieval rank), then the unseen 9
    assert O.recency_order([6, 9, 7, 5], m) == [7, 6, 5, 9]
    m1 = O.TreeModel(window=1)
    m1.insert([5, 6])
    m1.insert([7])
    assert O.recency_order([6, 9, 7, 5], m1) == [7, 6, 9, 5]


def test_oracle_greedy_equals_exhaustive_under_single_branch_condition():
    rng = np.random.default_rng(2)
    checked = 0
    for _ in range(300):
        k = int(rng.integers(2, 7))
        m = O.TreeModel(window=4)
        for _ in range(int(rng.integers(1, 6))):
            m.insert([int(x) for x in rng.permutation(9)[:int(rng.integers(1, 6))]])
        docs = [int(x) for x in rng.permutation(9)[:k]]
        order, depth, probes = O.greedy_order(docs, m.is_cached)
        assert sorted(order) == sorted(docs)
        assert probes <= k * (k + 1) // 2
        cached = _cached_orders(m)
        assert depth == O.walk_depth(order, m.is_cached) == O.reusable_prefix_depth(order, cached)
        best_order, best = O.exhaustive_order(docs, m.is_cached)
        # the k! search over the walk agrees with the one over the cached orders
        assert best == O.exhaustive_best_depth(docs, cached)
        assert best_order == O.canonical_best_order(docs, cached)[0]
        assert depth <= best
        if _single_branch(m, docs):
            checked += 1
            assert (order, depth) == (best_order, best)
    assert checked > 100


def test_oracle_greedy_can_trail_exhaustive_with_two_cached_children():
    m = O.TreeModel(window=8)
    m.insert([1, 5])          # shallow branch, first in retrieval rank
    m.insert([2, 3, 4])       # deeper branch
    assert O.greedy_order([1, 2, 3, 4], m.is_cached)[1] == 1
    assert O.exhaustive_order([1, 2, 3, 4], m.is_cached) == ([2, 3, 4, 1], 3)


def test_oracle_exhaustive_is_a_max_over_all_permutations():
    m = O.TreeModel(window=5)
    for o in ([1, 2, 3], [2, 1], [3, 4, 1, 2], [4]):
        m.insert(o)
    docs = [4, 1, 2, 3]
    best = max(O.walk_depth(p, m.is_cached) for p in itertools.permutations(docs))
    assert O.exhaustive_order(docs, m.is_cached)[1] == best == 4


# ---------------------------------------------------------------------------
# The library's tree against the oracle
# ---------------------------------------------------------------------------
def _expected(m, docs, strategy):
    if strategy == "greedy":
        return O.greedy_order(docs, m.is_cached)
    if strategy == "exhaustive":
        order, depth = O.exhaustive_order(docs, m.is_cached)
        return order, depth, None
    order = {"retrieval": O.retrieval_order(docs), "sorted": O.sorted_order(docs),
             "recency": O.recency_order(docs, m)}[strategy]
    return order, O.walk_depth(order, m.is_cached), None


STRATEGIES = ("retrieval", "sorted", "recency", "greedy", "exhaustive")


def test_tree_matches_oracle_on_random_histories():
    rng = np.random.default_rng(11)
    compared = 0
    for _ in range(150):
        window = int(rng.integers(1, 7))
        universe = int(rng.integers(3, 9))
        c, m = cw.KnowledgeTree(window), O.TreeModel(window)
        for _ in range(int(rng.integers(1, 30))):
            k = int(rng.integers(0, min(universe, 6) + 1))
            docs = [int(x) for x in rng.permutation(universe)[:k]]
            for s in STRATEGIES:
                got = c.order(docs, s)
                exp = _expected(m, docs, s)
                assert got[0] == list(exp[0]) and got[1] == exp[1], (s, docs)
                if exp[2] is not None:
                    assert got[2] == exp[2]
                compared += 1
            act = rng.random()
            if act < 0.6:                      # serve the greedy order, maybe with feedback
                o = c.order(docs, "greedy")[0]
                c.insert(o)
                m.insert(o)
                if o and rng.random() < 0.3:
                    obs = int(rng.integers(0, len(o) + 1))
                    c.mark_stale(o, obs)
                    m.mark_stale(o, obs)
            else:                              # an arbitrary order or a stray stale mark
                o = [int(x) for x in rng.permutation(universe)[:int(rng.integers(0, universe + 1))]]
                if act < 0.8:
                    c.insert(o)
                    m.insert(o)
                else:
                    obs = int(rng.integers(0, len(o) + 1))
                    c.mark_stale(o, obs)
                    m.mark_stale(o, obs)
        c.close()
    assert compared > 5000


def test_trace_orders_match_oracle():
    """The orders that shape the measured trace batch: libcw's tree and the
    oracle's greedy walk give the same order and depth for every query."""
    qs = W.synthetic_trace(80, pool_size=200, k=5, shared=3, seed=0)
    c, m = cw.KnowledgeTree(32), O.TreeModel(32)
    for docs in qs:
        got = c.order(docs)
        exp = O.greedy_order(docs, m.is_cached)
        assert got == exp
        c.insert(got[0])
        m.insert(exp[0])
    _, depths = W.serve_trace(qs, cw.KnowledgeTree(32), 256)
    assert sum(depths) > 0


def test_tree_fig2_example_and_probe_bound():
    ex = _fig2()
    t = cw.KnowledgeTree(window=8)
    t.insert([ord(x) for x in ex["cached_path"]])
    cand = [ord(x) for x in ex["candidates"]]
    order, depth, probes = t.order(cand)
    assert [chr(x) for x in order] == ex["expected_order"] and depth == int(ex["expected_depth"][0])
    assert probes <= len(cand) * (len(cand) + 1) // 2


def test_tree_space_bounded_by_window():
    t = cw.KnowledgeTree(window=8)
    for q in W.synthetic_trace(300, pool_size=50, k=5, shared=3, seed=1):
        t.insert(t.order(q)[0])
        assert t.num_nodes() <= 2 * 8 * 5


def test_tree_large_sets():
    t = cw.KnowledgeTree(window=4)
    big = list(range(10**12, 10**12 + 4096))
    t.insert(big)
    order, depth, _ = t.order(big[::-1], "greedy")
    assert order == big and depth == 4096                       # follows the one cached path
    order, depth, _ = t.order(big[::-1], "exhaustive")
    assert order == big and depth == 4096
    assert t.order(big[:100], "sorted")[1] == 100


def test_tree_rejects_bad_arguments():
    with pytest.raises(cw.CwError):
        cw.KnowledgeTree(window=0)
    t = cw.KnowledgeTree(window=4)
    for call in (lambda: t.insert([1, 1]), lambda: t.order([2, 3, 2]), lambda: t.order([1], 9),
                 lambda: t.mark_stale([1, 2], 3), lambda: t.mark_stale([1, 2], -1),
                 lambda: t.insert(range(4097))):
        with pytest.raises(cw.CwError) as e:
            call()
        assert e.value.status == cw.CW_EINVAL
    assert t.num_nodes() == 0
