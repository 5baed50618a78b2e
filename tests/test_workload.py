"""Host-side workload shaping: the synthetic trace's sharing model, the prompt
layout and the named batch shapes. (The ordering itself is tested in
test_ordering.py.)"""
import math

import numpy as np

from paper_2606_19667_amd import workload as W


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
