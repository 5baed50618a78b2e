"""Trace replay: the ordering side of the path, one request at a time.

For each query of a trace: order its retrieved set with the knowledge tree
(paper Sec. 3.3, Algorithm 1, or a baseline of Sec. 4), build the prompt
(instruction, ordered chunks, question; Sec. 4, prompt format), schedule it on
the block pool (chained hashes, prefix match, allocation, commit; Sec. 2.1),
release its blocks once served, and record the served order in the tree
(Sec. 3.2). With `feedback`, a request whose pool match reused fewer documents
than the tree predicted marks the deeper part of its path stale (Sec. 3.4).

The per-request record gives the prefill-saved proxy of Table `cache_eff`:
cached prompt tokens over prompt tokens, the no-cache prefill being the
shared denominator. A tight pool (fewer blocks than the recency window's
prompts need) evicts blocks the tree still believes resident, which is the
gap between the tree and true residency that Sec. 3.4 discusses.
"""
from __future__ import annotations

import math
import time
from dataclasses import dataclass, field

import numpy as np

from . import cw
from . import workload as W


@dataclass
class Replay:
    strategy: str
    feedback: bool
    num_blocks: int
    orders: list = field(default_factory=list)
    prompt_tokens: list = field(default_factory=list)
    cached_tokens: list = field(default_factory=list)
    predicted_docs: list = field(default_factory=list)   # l(O, T) of the chosen order
    reused_docs: list = field(default_factory=list)      # whole chunks inside the pool match
    order_ns: list = field(default_factory=list)
    schedule_ns: list = field(default_factory=list)

    def saved(self, skip: int = 0) -> np.ndarray:
        return (np.asarray(self.cached_tokens[skip:], np.float64)
                / np.asarray(self.prompt_tokens[skip:], np.float64))

    def summary(self, skip: int = 0) -> dict:
        """Prefill-saved fraction (p50 / mean / p95), requests that reused at
        least one evidence chunk, tree predictions the pool did not honour, and
        host time per request, over the requests after the first `skip`."""
        s = self.saved(skip)
        pred = np.asarray(self.predicted_docs[skip:])
        got = np.asarray(self.reused_docs[skip:])
        n = len(s)
        return {
            "requests": n,
            "saved_p50": round(float(np.percentile(s, 50)), 4) if n else None,
            "saved_mean": round(float(s.mean()), 4) if n else None,
            "saved_p95": round(float(np.percentile(s, 95)), 4) if n else None,
            "benefit": int((got > 0).sum()),
            "reused_docs_mean": round(float(got.mean()), 3) if n else None,
            "predicted_docs_mean": round(float(pred.mean()), 3) if n else None,
            "mispredicted": int((pred > got).sum()),
            "order_us": round(float(np.median(self.order_ns[skip:])) / 1e3, 2) if n else None,
            "schedule_us": round(float(np.median(self.schedule_ns[skip:])) / 1e3, 2) if n else None,
        }


def pool_blocks_for(queries, chunk_tokens: int, block_size: int = cw.BLOCK_SIZE) -> int:
    """Blocks for every prompt of the trace at once: nothing is ever evicted."""
    L = W.INSTR_TOKENS + W.QUESTION_TOKENS + chunk_tokens * max((len(q) for q in queries), default=0)
    return len(queries) * math.ceil(L / block_size)


def replay(queries, strategy: str = "greedy", chunk_tokens: int = 256, window: int = 32,
           num_blocks: int | None = None, feedback: bool = False, seed: int = 0,
           uid0: int = 0) -> Replay:
    """Serves `queries` (retrieved sets in retrieval rank) one by one."""
    bs = cw.BLOCK_SIZE
    if num_blocks is None:
        num_blocks = pool_blocks_for(queries, chunk_tokens, bs)
    tree = cw.KnowledgeTree(window)
    pool = cw.Pool(num_blocks)
    rec = Replay(strategy, feedback, num_blocks)
    try:
        for n, docs in enumerate(queries):
            t0 = time.perf_counter_ns()
            order, predicted, _ = tree.order(docs, strategy)
            t1 = time.perf_counter_ns()
            toks = W.rag_prompt(uid0 + n, order, chunk_tokens).tokens(seed)
            stride = math.ceil(len(toks) / bs)
            t2 = time.perf_counter_ns()
            bt, pl, cu = cw.schedule_batch(pool, [toks], stride, bs)
            t3 = time.perf_counter_ns()
            P = int(pl[0])
            reused = max(0, (P - W.INSTR_TOKENS) // chunk_tokens)
            cw.release_batch(pool, bt, pl, cu, bs)
            tree.insert(order)
            if feedback and reused < predicted:
                tree.mark_stale(order, reused)
            rec.orders.append(order)
            rec.prompt_tokens.append(len(toks))
            rec.cached_tokens.append(P)
            rec.predicted_docs.append(predicted)
            rec.reused_docs.append(reused)
            rec.order_ns.append(t1 - t0)
            rec.schedule_ns.append(t3 - t2)
    finally:
        tree.close()
        pool.close()
    return rec
