"""Synthetic RAG workloads: prompt layout, evidence ordering and batch shapes.

The ordering side of CacheWeaver only decides which prefix of each prompt is
already cached; this module reproduces that shaping on the host:

* The library's knowledge tree (`cw.KnowledgeTree`: the trie of recently
  served document orders, Sec. 3.2, with the greedy walk of Sec. 3.3,
  Algorithm 1, and recency as the residency estimate, Sec. 3.4) orders each
  query of a trace.
* `synthetic_trace` draws retrieved top-k sets in which consecutive queries
  share evidence (Sec. 4, workload paragraph: bursty overlapping retrieval; the
  exact generator is not given, so the sharing model is a stated choice).
* Prompts follow the paper's layout (Sec. 4, prompt format): a fixed
  instruction, the ordered evidence chunks, then the question.
* The batch builders produce the shapes the attention path is measured on.

Everything here is host-side, untimed set-up. Token IDs and K/V/Q values come
from `inputs` through integer keys only.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

from . import cw, inputs

INSTR_TOKENS = 64
QUESTION_TOKENS = 64

SEG_INSTR = 0
SEG_DOC_BASE = 1
SEG_QUESTION_BASE = 1 << 30

TAG_TOK, TAG_K, TAG_V, TAG_Q, TAG_TRACE, TAG_PLACE = 1, 2, 3, 4, 5, 6


# --------------------------------------------------------------------------
# Retrieved sets of a synthetic trace
# --------------------------------------------------------------------------
def synthetic_trace(n_queries: int, pool_size: int = 200, k: int = 5, shared: int = 3,
                    seed: int = 0):
    """Retrieved sets (each in retrieval rank) of consecutive queries.

    Each query keeps `shared` documents chosen uniformly from the previous
    query's set and draws the other k - shared from the rest of the pool; its
    retrieval rank is a uniform shuffle.
    """
    r = inputs.rng((seed, TAG_TRACE, pool_size, k, shared))
    prev = r.choice(pool_size, size=k, replace=False)
    out = [[int(d) for d in prev]]
    everything = np.arange(pool_size)
    for _ in range(1, n_queries):
        keep = r.choice(prev, size=shared, replace=False)
        fresh = r.choice(np.setdiff1d(everything, prev), size=k - shared, replace=False)
        cur = np.concatenate([keep, fresh])
        r.shuffle(cur)
        out.append([int(d) for d in cur])
        prev = cur
    return out


def jaccard(a, b) -> float:
    a, b = set(a), set(b)
    return len(a & b) / len(a | b) if (a or b) else 1.0


# --------------------------------------------------------------------------
# Prompts and their content
# --------------------------------------------------------------------------
@dataclass
class Prompt:
    """Instruction, ordered evidence chunks, question: a list of (segment, length)."""
    uid: int
    segments: list = field(default_factory=list)

    @property
    def length(self) -> int:
        return sum(n for _, n in self.segments)

    def tokens(self, seed: int) -> np.ndarray:
        return np.concatenate([inputs.token_ids((seed, TAG_TOK, s, n), n)
                               for s, n in self.segments]).astype(np.int32)

    def block_keys(self, block_size: int):
        """One key per (possibly partial) block: the segments that start before the
        block ends, plus the block index. Equal keys mean equal token prefixes."""
        starts = np.cumsum([0] + [n for _, n in self.segments])[:-1]
        keys = []
        for b in range(math.ceil(self.length / block_size)):
            end = min(self.length, (b + 1) * block_size)
            segs = tuple(s for (s, _), st in zip(self.segments, starts) if st < end)
            keys.append(segs + (b,))
        return keys


def rag_prompt(uid: int, docs, chunk_tokens: int, instr_tokens: int = INSTR_TOKENS,
               question_tokens: int = QUESTION_TOKENS) -> Prompt:
    segs = [(SEG_INSTR, instr_tokens)]
    segs += [(SEG_DOC_BASE + int(d), chunk_tokens) for d in docs]
    segs.append((SEG_QUESTION_BASE + int(uid), question_tokens))
    return Prompt(uid=uid, segments=segs)


@dataclass
class Workload:
    """A batch to prefill plus the requests served before it.

    prefix_lens is None when the cached depth comes from prefix matching on a
    block pool (trace workloads); otherwise it fixes each request's depth.
    content: "blocks" keys K/V/Q by block (requests with equal prefixes see equal
    values); "request" keys them by request (independent requests).
    """
    name: str
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    block_size: int
    prompts: list
    seed: int = 0
    prefix_lens: list | None = None
    content: str = "request"
    warmup: list = field(default_factory=list)
    trie_depths: list = field(default_factory=list)
    free_order_key: tuple = ()
    extra_blocks: int = 0

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    @property
    def batch(self) -> int:
        return len(self.prompts)

    def num_blocks(self) -> int:
        need = sum(math.ceil(p.length / self.block_size) for p in self.warmup + self.prompts)
        return need + self.extra_blocks

    def free_order(self) -> np.ndarray:
        return inputs.permutation((self.seed, TAG_PLACE) + tuple(self.free_order_key),
                                  self.num_blocks())


def logical_kv(w: Workload, prompt: Prompt, device="cpu"):
    """Logical K and V of a whole prompt: two [L, Hkv, D] bfloat16 tensors."""
    shape = (w.num_kv_heads, w.head_dim)
    if w.content == "request":
        k = inputs.normal_bf16((w.seed, TAG_K, prompt.uid), (prompt.length,) + shape, device)
        v = inputs.normal_bf16((w.seed, TAG_V, prompt.uid), (prompt.length,) + shape, device)
        return k, v
    ks, vs = [], []
    for b, key in enumerate(prompt.block_keys(w.block_size)):
        n = min(w.block_size, prompt.length - b * w.block_size)
        ks.append(inputs.normal_bf16((w.seed, TAG_K) + key, (n,) + shape, device))
        vs.append(inputs.normal_bf16((w.seed, TAG_V) + key, (n,) + shape, device))
    return torch.cat(ks), torch.cat(vs)


def suffix_q(w: Workload, prompt: Prompt, prefix_len: int, device="cpu"):
    """Queries of the suffix rows [prefix_len, L): [S, Hq, D] bfloat16."""
    shape = (w.num_q_heads, w.head_dim)
    if w.content == "request":
        q = inputs.normal_bf16((w.seed, TAG_Q, prompt.uid), (prompt.length,) + shape, device)
        return q[prefix_len:].contiguous()
    first = prefix_len // w.block_size
    qs = []
    keys = prompt.block_keys(w.block_size)
    for b in range(first, len(keys)):
        n = min(w.block_size, prompt.length - b * w.block_size)
        qs.append(inputs.normal_bf16((w.seed, TAG_Q) + keys[b], (n,) + shape, device))
    q = torch.cat(qs)
    return q[prefix_len - first * w.block_size:].contiguous()


# --------------------------------------------------------------------------
# Batches named by shape
# --------------------------------------------------------------------------
def tiny_single(seed: int = 0) -> Workload:
    """4 query heads, 1 KV head, head_dim 64, 16-token blocks; 64 cached prefix
    tokens (4 blocks) and a 32-token suffix; 8 physical blocks in random order."""
    p = Prompt(uid=0, segments=[(SEG_INSTR, 64), (SEG_QUESTION_BASE, 32)])
    return Workload("tiny-4q1kv-d64-p64-s32", 4, 1, 64, 16, [p], seed=seed,
                    prefix_lens=[64], extra_blocks=2)


def llama8b_single(seed: int = 0) -> Workload:
    """One Llama-3-8B-shaped request: 64-token instruction, 5 chunks of 256, 64-token
    question (1408 tokens); instruction + first 3 chunks cached (832), suffix 576."""
    p = rag_prompt(0, [0, 1, 2, 3, 4], 256)
    return Workload("llama8b-single-p832-s576", 32, 8, 128, 16, [p], seed=seed,
                    prefix_lens=[832])


def question_only(seed: int = 0, batch: int = 16) -> Workload:
    """`batch` Llama-3-8B-shaped requests whose whole evidence prefix is cached
    (instruction + 5 chunks of 256 = 1344 tokens): only the 64-token question is
    prefilled. The deepest reuse the ordering aims for; a short-suffix shape."""
    prompts = [rag_prompt(r, range(5 * r, 5 * r + 5), 256) for r in range(batch)]
    P = INSTR_TOKENS + 5 * 256
    return Workload(f"llama8b-question-only-b{batch}-p{P}-s{QUESTION_TOKENS}", 32, 8, 128, 16, prompts,
                    seed=seed, prefix_lens=[P] * batch, free_order_key=(64,))


def serve_trace(queries, tree: "cw.KnowledgeTree", chunk_tokens: int, uid0: int = 0):
    """Order each query with the tree, insert it after serving; returns prompts
    and the greedy depth (documents) of each."""
    prompts, depths = [], []
    for n, docs in enumerate(queries):
        order, depth, _ = tree.order(docs)
        prompts.append(rag_prompt(uid0 + n, order, chunk_tokens))
        depths.append(depth)
        tree.insert(order)
    return prompts, depths


def llama8b_trace_batch(seed: int = 0, batch: int = 16, warmup: int = 64,
                        pool_size: int = 200, k: int = 5, shared: int = 3,
                        chunk_tokens: int = 256, window: int = 32) -> Workload:
    """A batch of `batch` consecutive queries of a synthetic trace (pool of 200
    chunks of 256 tokens, top-5, 3 of 5 chunks shared with the previous query)
    ordered by the greedy tree walk, after `warmup` served queries; 8B-shaped
    heads. Cached depths follow from prefix matching the pool."""
    qs = synthetic_trace(warmup + batch, pool_size, k, shared, seed)
    tree = cw.KnowledgeTree(window)
    prompts, depths = serve_trace(qs, tree, chunk_tokens)
    return Workload(f"llama8b-trace-b{batch}-k{k}-share{shared}of{k}", 32, 8, 128, 16,
                    prompts[warmup:], seed=seed, content="blocks",
                    warmup=prompts[:warmup], trie_depths=depths[warmup:])


def topk_sweep(frac: float, seed: int = 0, batch: int = 8) -> Workload:
    """k = 10 chunks of 512 tokens + 64-token instruction + 64-token question
    (5248 tokens), `batch` requests, a fixed cached fraction of blocks."""
    L = INSTR_TOKENS + 10 * 512 + QUESTION_TOKENS
    nb = math.ceil(L / 16)
    P = int(math.floor(frac * nb)) * 16
    prompts = [rag_prompt(r, range(10 * r, 10 * r + 10), 512) for r in range(batch)]
    return Workload(f"topk10-L{L}-b{batch}-f{frac:g}", 32, 8, 128, 16, prompts, seed=seed,
                    prefix_lens=[P] * batch, free_order_key=(int(frac * 100),))


def long_context(hit: str, seed: int = 0, batch: int = 64) -> Workload:
    """70B-shaped heads (64 Q, 8 KV), k = 20 chunks of 512 tokens + 64 + 64
    (10368 tokens), `batch` requests; cached depth of l_r whole chunks drawn
    uniformly from 0..4 ("low", ~10 % of tokens) or 12..16 ("high", ~70 %)."""
    L = INSTR_TOKENS + 20 * 512 + QUESTION_TOKENS
    lo, hi = (0, 4) if hit == "low" else (12, 16)
    r = inputs.rng((seed, TAG_TRACE, 70, lo, hi))
    depths = r.integers(lo, hi + 1, size=batch)
    prompts = [rag_prompt(i, range(20 * i, 20 * i + 20), 512) for i in range(batch)]
    P = [INSTR_TOKENS + 512 * int(d) for d in depths]
    return Workload(f"llama70b-long-L{L}-b{batch}-{hit}", 64, 8, 128, 16, prompts, seed=seed,
                    prefix_lens=P, free_order_key=(hi,))
