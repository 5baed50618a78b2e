"""Trace replay (CPU): the ordering side of the path, request by request.

The library's replay (knowledge tree + block pool, both native) is compared
with the same loop built from oracle parts only: the oracle tree model and its
orders, chained XXH64 block hashes and the pool simulation. Orders, cached
prefix lengths, predicted and reused depths must match exactly, for every
strategy with an unbounded pool, and for a pool too small for the recency
window, with and without stale-path feedback.
"""
import math

import numpy as np
import pytest

from oracle import ordering as O
from oracle import paged
from paper_2606_19667_amd import cw
from paper_2606_19667_amd import replay as R
from paper_2606_19667_amd import workload as W


def _oracle_replay(queries, strategy, chunk_tokens=256, window=32, num_blocks=None,
                   feedback=False, seed=0):
    bs = 16
    if num_blocks is None:
        num_blocks = R.pool_blocks_for(queries, chunk_tokens, bs)
    tree = O.TreeModel(window)
    pool = paged.PoolSim(num_blocks)
    out = []
    for n, docs in enumerate(queries):
        if strategy == "greedy":
            order = O.greedy_order(docs, tree.is_cached)[0]
        elif strategy == "exhaustive":
            order = O.exhaustive_order(docs, tree.is_cached)[0]
        elif strategy == "recency":
            order = O.recency_order(docs, tree)
        elif strategy == "sorted":
            order = O.sorted_order(docs)
        else:
            order = O.retrieval_order(docs)
        predicted = O.walk_depth(order, tree.is_cached)
        toks = W.rag_prompt(n, order, chunk_tokens).tokens(seed)
        hs = paged.chain_block_hashes(toks, bs)
        ids = pool.prefix_match(hs, (len(toks) - 1) // bs)
        new = pool.alloc(math.ceil(len(toks) / bs) - len(ids))
        pool.commit(hs[len(ids):], new[:len(hs) - len(ids)])
        P = len(ids) * bs
        pool.release(ids + new)
        reused = max(0, (P - W.INSTR_TOKENS) // chunk_tokens)
        tree.insert(order)
        if feedback and reused < predicted:
            tree.mark_stale(order, reused)
        out.append((list(order), P, predicted, reused))
    return out


def _check(rec, exp):
    got = list(zip(rec.orders, rec.cached_tokens, rec.predicted_docs, rec.reused_docs))
    assert len(got) == len(exp)
    for i, (g, e) in enumerate(zip(got, exp)):
        assert g == e, f"request {i}: {g} != {e}"


@pytest.mark.parametrize("strategy", ["retrieval", "sorted", "recency", "greedy", "exhaustive"])
def test_replay_matches_oracle_unbounded_pool(strategy):
    qs = W.synthetic_trace(60, pool_size=200, k=5, shared=3, seed=0)
    _check(R.replay(qs, strategy), _oracle_replay(qs, strategy))


@pytest.mark.parametrize("feedback", [False, True])
def test_replay_matches_oracle_tight_pool(feedback):
    qs = W.synthetic_trace(100, pool_size=60, k=5, shared=3, seed=3)
    nb = 4 * 88                     # four 1408-token prompts for a 32-order window
    rec = R.replay(qs, "greedy", num_blocks=nb, feedback=feedback)
    _check(rec, _oracle_replay(qs, "greedy", num_blocks=nb, feedback=feedback))
    if not feedback:
        # the tree believes in paths the pool has evicted
        assert rec.summary()["mispredicted"] > 0


def test_replay_proxy_invariants():
    qs = W.synthetic_trace(120, pool_size=200, k=5, shared=3, seed=1)
    recs = {s: R.replay(qs, s) for s in ("retrieval", "greedy", "exhaustive")}
    for s, rec in recs.items():
        saved = rec.saved()
        assert ((saved >= 0) & (saved < 1)).all()
        # an unbounded pool honours every prediction; the instruction is always shared
        assert rec.summary()["mispredicted"] == 0
        assert all(p >= W.INSTR_TOKENS for p in rec.cached_tokens[1:])
    assert recs["greedy"].saved().mean() > recs["retrieval"].saved().mean()
    # on one tree state the exhaustive search never predicts less than the walk
    tree = cw.KnowledgeTree(32)
    for docs in qs:
        g = tree.order(docs, "greedy")
        assert tree.order(docs, "exhaustive")[1] >= g[1]
        tree.insert(g[0])
