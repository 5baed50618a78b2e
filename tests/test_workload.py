"""Host-side workload shaping: the greedy tree walk against the paper's example,
its fallback and its optimality condition (checked against the exhaustive
search of oracle.ordering), and the synthetic prompt layout."""
import itertools
import math
import os

import numpy as np
import pytest

from oracle import ordering
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


def test_fig2_example():
    ex = _fig2()
    t = W.KnowledgeTree(window=8)
    t.insert(ex["cached_path"])
    order, depth, probes = t.order(ex["candidates"])
    assert order == ex["expected_order"]
    assert depth == int(ex["expected_depth"][0])
    assert ordering.reusable_prefix_depth(order, [ex["cached_path"]]) == depth
    k = len(ex["candidates"])
    assert probes <= k * (k + 1) // 2


def test_fallback_is_retrieval_order():
    t = W.KnowledgeTree(window=4)
    assert t.order([5, 3, 9])[0] == [5, 3, 9]          # empty tree
    t.insert([1, 2, 3])
    assert t.order([7, 8, 2])[:2] == ([7, 8, 2], 0)     # no cached continuation from the root


def test_recency_window_expires_paths():
    t = W.KnowledgeTree(window=3)
    t.insert([1, 2])
    for n in range(3):
        t.insert([10 + n])
    assert t.order([2, 1])[1] == 0                      # served 4 requests ago: not cached
    t.insert([1, 2])
    assert t.order([2, 1]) == ([1, 2], 2, 3)   # root: 2 misses, 1 hits; then 2 hits


def _single_branch(tree, docs):
    """Every node the walk can visit has at most one cached child still in R."""
    stack = [(tree.root, set(docs))]
    while stack:
        node, rem = stack.pop()
        kids = [(d, c) for d, c in node.children.items() if d in rem and tree.is_cached(c)]
        if len(kids) > 1:
            return False
        for d, c in kids:
            stack.append((c, rem - {d}))
    return True


def test_greedy_equals_exhaustive_under_single_branch_condition():
    rng = np.random.default_rng(2)
    checked = 0
    for trial in range(400):
        k = int(rng.integers(2, 7))
        universe = list(range(9))
        t = W.KnowledgeTree(window=4)
        served = []
        for _ in range(int(rng.integers(1, 6))):
            o = [int(x) for x in rng.permutation(universe)[:int(rng.integers(1, 6))]]
            t.insert(o)
            served.append(o)
        docs = [int(x) for x in rng.permutation(universe)[:k]]
        cached = served[-4:]
        order, depth, probes = t.order(docs)
        assert sorted(order) == sorted(docs)
        assert probes <= k * (k + 1) // 2
        assert depth == ordering.reusable_prefix_depth(order, cached)
        best = ordering.exhaustive_best_depth(docs, cached)
        assert depth <= best
        if _single_branch(t, docs):
            checked += 1
            assert depth == best
            assert order == ordering.canonical_best_order(docs, cached)[0]
    assert checked > 100


def test_greedy_can_trail_exhaustive_with_two_cached_children():
    t = W.KnowledgeTree(window=8)
    t.insert([1, 5])            # shallow branch, first in retrieval rank
    t.insert([2, 3, 4])         # deeper branch
    order, depth, _ = t.order([1, 2, 3, 4])
    assert depth == 1 and ordering.exhaustive_best_depth([1, 2, 3, 4], [[1, 5], [2, 3, 4]]) == 3


def test_tree_space_bounded_by_window():
    t = W.KnowledgeTree(window=8)
    for q in W.synthetic_trace(300, pool_size=50, k=5, shared=3, seed=1):
        t.insert(t.order(q)[0])
    assert t.num_nodes() <= 2 * 8 * 5


def test_trace_sharing_model():
    qs = W.synthetic_trace(50, pool_size=200, k=5, shared=3, seed=0)
    for a, b in zip(qs, qs[1:]):
        assert len(set(a) & set(b)) == 3 and len(set(b)) == 5
        assert abs(W.jaccard(a, b) - 3 / 7) < 1e-12


def test_prompt_layout_and_block_keys():
    p = W.rag_prompt(7, [3, 1], 256)
    assert p.length == 64 + 512 + 64
    toks = p.tokens(0)
    q = W.rag_prompt(8, [3, 2], 256)
    # the same instruction and first document give the same tokens and keys
    assert np.array_equal(toks[:64 + 256], q.tokens(0)[:64 + 256])
    assert p.block_keys(16)[:20] == q.block_keys(16)[:20]
    assert p.block_keys(16)[20] != q.block_keys(16)[20]
    assert len(p.block_keys(16)) == math.ceil(p.length / 16)


def test_named_shapes():
    w = W.tiny_single()
    assert (w.num_q_heads, w.num_kv_heads, w.head_dim, w.prompts[0].length, w.prefix_lens) == (4, 1, 64, 96, [64])
    assert w.num_blocks() == 8
    w = W.llama8b_single()
    assert w.prompts[0].length == 1408 and w.prefix_lens == [832]
    w = W.topk_sweep(0.6)
    assert w.prompts[0].length == 5248 and w.prefix_lens[0] == 196 * 16
    w = W.long_context("high")
    assert w.prompts[0].length == 10368
    assert all(64 + 512 * 12 <= p <= 64 + 512 * 16 for p in w.prefix_lens)


def test_question_only_shape():
    w = W.question_only()
    assert w.batch == 16 and all(p.length == 1408 for p in w.prompts)
    assert w.prefix_lens == [1344] * 16
    # the 4 instruction blocks are common; every later block is the request's own
    keys = [p.block_keys(16) for p in w.prompts]
    assert all(k[:4] == keys[0][:4] for k in keys)
    later = [set(k[4:]) for k in keys]
    assert all(not (later[a] & later[b]) for a in range(16) for b in range(a + 1, 16))
