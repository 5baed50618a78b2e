"""Pins of the CPU oracle to things other than itself.

Attention: brute-force loops, torch's fp64 scaled_dot_product_attention with an
explicit mask, closed forms, a hand-worked example, the GQA mapping and the
prefix-cached == from-scratch invariant. Hashing: published XXH64 values and
the xxhash library. Pool and append: brute force on tokens, the paper's Fig. 1
scenario, hand-worked examples.
"""
import math
import os
import struct

import numpy as np
import pytest
import torch

from oracle import attention as A
from oracle import paged

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _rand(shape, seed):
    return np.random.default_rng(seed).standard_normal(shape)


def _case(S, P, Hq, Hkv, D, seed):
    q = _rand((S, Hq, D), seed)
    k = _rand((P + S, Hkv, D), seed + 1)
    v = _rand((P + S, Hkv, D), seed + 2)
    return q, k, v


# ---------------------------------------------------------------- attention
@pytest.mark.parametrize("S,P,Hq,Hkv,D", [(1, 0, 1, 1, 4), (3, 5, 4, 2, 8), (7, 16, 4, 1, 16),
                                          (5, 0, 8, 2, 8), (2, 33, 2, 2, 4)])
def test_vectorized_matches_loops(S, P, Hq, Hkv, D):
    q, k, v = _case(S, P, Hq, Hkv, D, 11 * S + P)
    a = A.suffix_prefill_attention(q, k, v, P, 1 / math.sqrt(D))
    b = A.suffix_prefill_attention_loops(q, k, v, P, 1 / math.sqrt(D))
    assert np.max(np.abs(a - b)) <= 1e-12


def test_tiny_config_matches_loops():
    """4 Q heads, 1 KV head, D 64, P 64, S 32 in bf16 values (upcast exactly)."""
    g = torch.Generator().manual_seed(3)
    q = torch.randn(32, 4, 64, generator=g).to(torch.bfloat16)
    k = torch.randn(96, 1, 64, generator=g).to(torch.bfloat16)
    v = torch.randn(96, 1, 64, generator=g).to(torch.bfloat16)
    a = A.suffix_prefill_attention(q, k, v, 64, 0.125)
    b = A.suffix_prefill_attention_loops(q, k, v, 64, 0.125)
    assert np.max(np.abs(a - b)) <= 1e-12


@pytest.mark.parametrize("S,P,Hq,Hkv,D", [(9, 0, 4, 1, 16), (9, 23, 8, 2, 32), (40, 48, 32, 8, 64)])
def test_matches_torch_sdpa_fp64(S, P, Hq, Hkv, D):
    q, k, v = _case(S, P, Hq, Hkv, D, 5 + S)
    scale = 1 / math.sqrt(D)
    got = A.suffix_prefill_attention(q, k, v, P, scale)
    G = Hq // Hkv
    qt = torch.from_numpy(q).permute(1, 0, 2)[None]
    kt = torch.from_numpy(k).repeat_interleave(G, dim=1).permute(1, 0, 2)[None]
    vt = torch.from_numpy(v).repeat_interleave(G, dim=1).permute(1, 0, 2)[None]
    mask = torch.arange(P + S)[None, :] <= (P + torch.arange(S))[:, None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, attn_mask=mask, scale=scale)
    ref = ref[0].permute(1, 0, 2).numpy()
    assert np.max(np.abs(got - ref)) <= 1e-10
    if P == 0:
        ref2 = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, scale=scale)
        assert np.max(np.abs(got - ref2[0].permute(1, 0, 2).numpy())) <= 1e-10


@pytest.mark.parametrize("P,S", [(16, 8), (64, 32), (0, 12)])
def test_prefix_cached_equals_full_prefill(P, S):
    q_full, k, v = _case(P + S, 0, 4, 2, 16, 77)
    full = A.suffix_prefill_attention(q_full, k, v, 0, 0.25)
    part = A.suffix_prefill_attention(q_full[P:], k, v, P, 0.25)
    assert np.max(np.abs(full[P:] - part)) <= 1e-12


def test_constant_values_give_that_constant():
    q, k, v = _case(6, 10, 4, 2, 8, 1)
    c = np.array([[1.5, -2, 0.25, 3, 0, 7, -1, 2], [0.5, 0.5, -4, 1, 1, 1, 9, -3]])
    v[:] = c[None]
    out = A.suffix_prefill_attention(q, k, v, 10, 0.3)
    for h in range(4):
        assert np.max(np.abs(out[:, h] - c[h // 2][None])) <= 1e-12


def test_zero_query_averages_visible_values():
    q, k, v = _case(5, 7, 2, 1, 4, 2)
    q[:] = 0
    out = A.suffix_prefill_attention(q, k, v, 7, 1.0)
    for i in range(5):
        expect = v[:7 + i + 1, 0].mean(axis=0)
        for h in range(2):
            assert np.max(np.abs(out[i, h] - expect)) <= 1e-12


def test_single_row_no_prefix_returns_first_value():
    q, k, v = _case(1, 0, 4, 4, 8, 3)
    out = A.suffix_prefill_attention(q, k, v, 0, 0.35)
    assert np.max(np.abs(out[0] - v[0])) <= 1e-15


def test_dominant_logit_selects_its_value():
    q, k, v = _case(1, 9, 1, 1, 4, 4)
    q[0, 0] = [10.0, 0, 0, 0]
    k[:] = 0
    k[5, 0] = [10.0, 0, 0, 0]
    out = A.suffix_prefill_attention(q, k, v, 9, 1.0)
    assert np.max(np.abs(out[0, 0] - v[5, 0])) <= 1e-30 + 1e-40 + 9 * math.exp(-100) * 10


def test_hand_worked_two_keys():
    """P = 1, S = 1, D = 64, scale 1/8: q.k0 = 8 (logit 1), q.k1 = 0 (logit 0), so
    O = (e v0 + v1) / (e + 1)."""
    D = 64
    q = np.zeros((1, 1, D)); q[0, 0, 0] = 2.0
    k = np.zeros((2, 1, D)); k[0, 0, 0] = 4.0; k[1, 0, 1] = 5.0
    v = np.zeros((2, 1, D)); v[0, 0, :] = 1.0; v[1, 0, :] = -1.0; v[1, 0, 3] = 10.0
    out = A.suffix_prefill_attention(q, k, v, 1, 1 / 8)
    e = math.e
    expect = (e * v[0, 0] + v[1, 0]) / (e + 1)
    assert np.max(np.abs(out[0, 0] - expect)) <= 1e-15


def test_gqa_uses_contiguous_groups():
    """Hq 4, Hkv 2: heads 0,1 read KV head 0 and heads 2,3 read KV head 1 (not h % Hkv)."""
    q, k, v = _case(3, 4, 4, 2, 8, 9)
    v[:, 0, :] = 1.0
    v[:, 1, :] = 2.0
    out = A.suffix_prefill_attention(q, k, v, 4, 0.3)
    assert np.allclose(out[:, 0], 1) and np.allclose(out[:, 1], 1)
    assert np.allclose(out[:, 2], 2) and np.allclose(out[:, 3], 2)


def test_future_keys_are_invisible_and_diagonal_is_visible():
    q, k, v = _case(6, 5, 2, 1, 8, 10)
    base = A.suffix_prefill_attention(q, k, v, 5, 0.3)
    k2, v2 = k.copy(), v.copy()
    k2[5 + 3:] = 99.0
    v2[5 + 3:] = -99.0
    pert = A.suffix_prefill_attention(q, k2, v2, 5, 0.3)
    assert np.max(np.abs(base[:3] - pert[:3])) == 0.0
    assert np.max(np.abs(base[3:] - pert[3:])) > 1.0   # row 3 sees key 8 = P + 3


def test_sampled_rows_equal_full_rows():
    q, k, v = _case(20, 16, 4, 2, 8, 12)
    full = A.suffix_prefill_attention(q, k, v, 16, 0.3)
    rows = [0, 7, 19]
    assert np.max(np.abs(A.suffix_prefill_rows(q, k, v, 16, 0.3, rows) - full[rows])) <= 1e-13


def test_row_chunking_does_not_change_rows():
    q, k, v = _case(37, 20, 4, 2, 8, 13)
    a = A.suffix_prefill_attention(q, k, v, 20, 0.3, row_chunk=5)
    b = A.suffix_prefill_attention(q, k, v, 20, 0.3, row_chunk=1000)
    assert np.max(np.abs(a - b)) <= 1e-14


def test_empty_suffix():
    q = np.zeros((0, 4, 8))
    k = _rand((16, 2, 8), 0)
    out = A.suffix_prefill_attention(q, k, k, 16, 0.3)
    assert out.shape == (0, 4, 8)


# ---------------------------------------------------------------- partial attention + merge
def _rand_qkv(rng, S, P, Hq, Hkv, D):
    return (rng.standard_normal((S, Hq, D)), rng.standard_normal((P + S, Hkv, D)),
            rng.standard_normal((P + S, Hkv, D)))


def _merge_parts(parts, S, Hq, D):
    o = np.stack([p[0].reshape(S * Hq, D) for p in parts])
    l = np.stack([p[1].reshape(S * Hq) for p in parts])
    return A.lse_merge(o, l).reshape(S, Hq, D)


@pytest.mark.parametrize("cuts", [[0, 64], [0, 3, 64], [0, 16, 17, 40, 64], [0, 30, 35, 64]])
def test_merge_of_key_partition_equals_full_attention(cuts):
    """Parts over disjoint key ranges that cover all keys merge to the full
    result; ranges past some rows' causal limit (empty parts) included."""
    rng = np.random.default_rng(len(cuts))
    S, P, Hq, Hkv, D = 10, 22, 4, 2, 8
    cuts = [min(c, P + S) for c in cuts]
    q, k, v = _rand_qkv(rng, S, P, Hq, Hkv, D)
    parts = [A.suffix_prefill_partial(q, k, v, P, 0.2, a, b) for a, b in zip(cuts[:-1], cuts[1:])]
    full = A.suffix_prefill_attention(q, k, v, P, 0.2)
    assert np.abs(_merge_parts(parts, S, Hq, D) - full).max() < 1e-12
    # the merge does not depend on the order of the parts
    assert np.abs(_merge_parts(parts[::-1], S, Hq, D) - full).max() < 1e-12


def test_single_part_is_full_attention_and_its_lse():
    """One part over every key: o is the full result and lse2 is the library
    log-sum-exp of the visible scaled scores, divided by ln 2."""
    from scipy.special import logsumexp
    rng = np.random.default_rng(3)
    S, P, Hq, Hkv, D = 5, 7, 2, 1, 4
    q, k, v = _rand_qkv(rng, S, P, Hq, Hkv, D)
    o, lse2 = A.suffix_prefill_partial(q, k, v, P, 0.5, 0, P + S)
    assert np.abs(o - A.suffix_prefill_attention(q, k, v, P, 0.5)).max() < 1e-12
    for i in range(S):
        for h in range(Hq):
            s = 0.5 * (k[:P + i + 1, 0, :] @ q[i, h, :])
            assert abs(lse2[i, h] - logsumexp(s) / math.log(2.0)) < 1e-12


def test_merge_two_keys_closed_form():
    s0, s1 = 0.7, -1.9
    v0, v1 = np.array([[1.0, -2.0]]), np.array([[3.0, 0.5]])
    lse = np.array([[s0 / math.log(2.0)], [s1 / math.log(2.0)]])
    got = A.lse_merge(np.stack([v0, v1]), lse)
    want = (math.exp(s0) * v0 + math.exp(s1) * v1) / (math.exp(s0) + math.exp(s1))
    assert np.abs(got - want).max() < 1e-14


def test_merge_skips_empty_parts_and_zeroes_empty_rows():
    o = np.array([[[1.0, 2.0], [5.0, 5.0]], [[9.0, 9.0], [7.0, 8.0]]])   # [2 parts, 2 rows, 2]
    lse = np.array([[3.0, -np.inf], [-np.inf, -np.inf]])
    got = A.lse_merge(o, lse)
    assert got[0].tolist() == [1.0, 2.0] and got[1].tolist() == [0.0, 0.0]


def test_partial_rows_past_the_part_are_empty():
    rng = np.random.default_rng(4)
    S, P = 4, 8
    q, k, v = _rand_qkv(rng, S, P, 2, 1, 4)
    o, lse2 = A.suffix_prefill_partial(q, k, v, P, 0.3, P + 2, P + S)   # keys P+2 .. P+3
    assert np.isneginf(lse2[:2]).all() and (o[:2] == 0).all()          # rows 0, 1 see none
    assert np.isfinite(lse2[2:]).all()


def test_flop_count_closed_form():
    # S = 2, P = 3: pairs = 2 * 3 + 3 = 9 (row 0 sees 4 keys, row 1 sees 5)
    assert A.attention_flops([3], [2], 1, 1) == 4 * 9


# ---------------------------------------------------------------- hashing
def _golden_vectors():
    rows = []
    with open(os.path.join(GOLDEN, "xxh64_vectors.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            seed, hexd, msg = line.split(maxsplit=2)
            rows.append((int(seed), int(hexd, 16), msg.strip()[1:-1].encode()))
    return rows


def test_xxh64_published_vectors():
    rows = _golden_vectors()
    assert rows
    for seed, digest, msg in rows:
        assert paged.xxh64(msg, seed) == digest


def test_xxh64_matches_library_all_tail_paths():
    xxhash = pytest.importorskip("xxhash")
    rng = np.random.default_rng(0)
    for n in list(range(0, 80)) + [127, 128, 129, 255, 1000]:
        data = rng.integers(0, 256, size=n, dtype=np.uint8).tobytes()
        for seed in (0, 1, 0xFFFFFFFFFFFFFFFF, int(rng.integers(0, 2**63))):
            assert paged.xxh64(data, seed) == xxhash.xxh64(data, seed=seed).intdigest()


def test_chain_hash_definition_and_prefix_sensitivity():
    xxhash = pytest.importorskip("xxhash")
    toks = np.arange(1000, 1000 + 16 * 5 + 7, dtype=np.int32)
    hs = paged.chain_block_hashes(toks, 16)
    assert len(hs) == 5                                   # the partial block has no hash
    h = 0
    for b in range(5):
        h = xxhash.xxh64(toks[16 * b:16 * b + 16].astype("<i4").tobytes(), seed=h).intdigest()
        assert hs[b] == h
    t2 = toks.copy()
    t2[20] += 1                                           # block 1 changes
    h2 = paged.chain_block_hashes(t2, 16)
    assert h2[0] == hs[0] and all(a != b for a, b in zip(h2[1:], hs[1:]))
    assert paged.chain_block_hashes(toks[:16 * 5], 16) == hs


# ---------------------------------------------------------------- pool
def _full_blocks_common(a, b, bs):
    n = 0
    while (n + 1) * bs <= min(len(a), len(b)) and np.array_equal(a[n * bs:(n + 1) * bs], b[n * bs:(n + 1) * bs]):
        n += 1
    return n


def test_prefix_match_equals_brute_force_on_tokens():
    rng = np.random.default_rng(5)
    bs = 4
    alphabet = [rng.integers(0, 50, size=bs * 3, dtype=np.int32) for _ in range(6)]
    pool = paged.PoolSim(4000)
    served = []
    for n in range(60):
        docs = rng.permutation(6)[:rng.integers(1, 5)]
        toks = np.concatenate([alphabet[0][:bs]] + [alphabet[d] for d in docs]
                              + [rng.integers(0, 50, size=rng.integers(1, 9), dtype=np.int32)])
        hs = paged.chain_block_hashes(toks, bs)
        cap = (len(toks) - 1) // bs
        ids = pool.prefix_match(hs, cap)
        brute = max([_full_blocks_common(toks, s, bs) for s in served] + [0])
        assert len(ids) == min(brute, cap)
        new = pool.alloc(math.ceil(len(toks) / bs) - len(ids))
        table = ids + new
        pool.commit(hs[len(ids):], table[len(ids):len(hs)])
        pool.release(table)
        served.append(toks)


def test_fig1_scenario_reorder_restores_prefix():
    """Request 2 shares 4 of request 1's 5 documents; in retrieval order its first
    document differs, so only the instruction matches; putting the shared
    documents first in request 1's order matches them too (paper Fig. 1)."""
    bs = 16
    instr = np.arange(64, dtype=np.int32)
    doc = {d: np.full(32, 1000 + d, dtype=np.int32) + np.arange(32, dtype=np.int32) for d in range(10)}

    def prompt(order, qid):
        return np.concatenate([instr] + [doc[d] for d in order] + [np.full(16, 5000 + qid, dtype=np.int32)])

    pool = paged.PoolSim(200)
    p1 = prompt([1, 2, 3, 4, 5], 1)
    h1 = paged.chain_block_hashes(p1, bs)
    t1 = pool.alloc(len(h1))
    pool.commit(h1, t1)
    pool.release(t1)
    retrieval = prompt([9, 1, 2, 3, 4], 2)
    assert len(pool.prefix_match(paged.chain_block_hashes(retrieval, bs), 100)) == 4   # instruction only
    pool2 = paged.PoolSim(200)
    t = pool2.alloc(len(h1)); pool2.commit(h1, t); pool2.release(t)
    reordered = prompt([1, 2, 3, 4, 9], 2)
    assert len(pool2.prefix_match(paged.chain_block_hashes(reordered, bs), 100)) == 4 + 4 * 2


def test_pool_alloc_order_eviction_and_errors():
    pool = paged.PoolSim(4, free_order=[2, 0, 3, 1])
    a = pool.alloc(2)
    assert a == [2, 0]
    pool.commit([111, 222], a)
    pool.release(a)                      # reverse order: 0 then 2 join the back
    assert pool.free == [3, 1, 0, 2]
    assert pool.prefix_match([111, 222, 333], 3) == [2, 0]
    assert pool.free == [3, 1]
    with pytest.raises(ValueError):
        pool.alloc(3)                    # no state change on failure
    assert pool.free == [3, 1]
    pool.release([2, 0])                 # reverse order: 0 joins the back, then 2
    assert pool.free == [3, 1, 0, 2]
    b = pool.alloc(3)                    # 3, 1 fresh, then 0 (holding 222) is evicted
    assert b == [3, 1, 0] and 222 not in pool.table and pool.table[111] == 2
    assert pool.prefix_match([111, 222], 2) == [2]
    with pytest.raises(ValueError):
        pool.release([2, 2])             # 2 is held once
    pool.release([2])
    with pytest.raises(ValueError):
        pool.commit([5], [2])            # commit needs a held block
    pool.commit([999], [3])
    pool.commit([999], [1])              # duplicate hash: first block stays
    assert pool.table[999] == 3 and pool.hash_of[1] is None


# ---------------------------------------------------------------- append image
def test_append_image_hand_example():
    cache = np.zeros((4, 1, 4, 2), dtype=np.uint16)
    new = np.arange(1, 1 + 5 * 1 * 2, dtype=np.uint16).reshape(5, 1, 2)
    bt = np.array([[3, 1, 0]], dtype=np.int32)
    out = paged.kv_append_image(cache, new, bt, [0, 5], [4], block_size=4)
    # tokens 4..7 -> block 1 slots 0..3, token 8 -> block 0 slot 0
    assert out[1, 0].tolist() == [[1, 2], [3, 4], [5, 6], [7, 8]]
    assert out[0, 0, 0].tolist() == [9, 10] and out[0, 0, 1:].sum() == 0
    assert out[3].sum() == 0 and out[2].sum() == 0


def test_append_image_transposed_hand_example():
    cache = np.zeros((4, 1, 2, 4), dtype=np.uint16)      # [NB, Hkv, D, bs]
    new = np.arange(1, 1 + 5 * 1 * 2, dtype=np.uint16).reshape(5, 1, 2)
    bt = np.array([[3, 1, 0]], dtype=np.int32)
    out = paged.kv_append_image(cache, new, bt, [0, 5], [4], block_size=4, layout="d_slot")
    # tokens 4..7 -> block 1 slots 0..3: d = 0 row holds 1, 3, 5, 7; d = 1 row 2, 4, 6, 8
    assert out[1, 0].tolist() == [[1, 3, 5, 7], [2, 4, 6, 8]]
    assert out[0, 0, :, 0].tolist() == [9, 10] and out[0, 0, :, 1:].sum() == 0
    assert out[3].sum() == 0 and out[2].sum() == 0
    with pytest.raises(ValueError):
        paged.kv_append_image(cache, new, bt, [0, 5], [4], block_size=4, layout="dslot")


@pytest.mark.parametrize("layout", ["slot_d", "d_slot"])
def test_append_image_vectorized_matches_loops(layout):
    rng = np.random.default_rng(8)
    shape = (12, 2, 4, 3) if layout == "slot_d" else (12, 2, 3, 4)
    cache = rng.integers(0, 65535, size=shape, dtype=np.uint16)
    P = [4, 0, 8]
    S = [5, 3, 1]
    cu = np.concatenate([[0], np.cumsum(S)])
    new = rng.integers(0, 65535, size=(cu[-1], 2, 3), dtype=np.uint16)
    bt = np.array([[0, 5, 7, 11], [2, 3, 1, 1], [9, 10, 4, 4]], dtype=np.int32)
    a = paged.kv_append_image(cache, new, bt, cu, P, 4, layout=layout)
    b = paged.kv_append_image_loops(cache, new, bt, cu, P, 4, layout=layout)
    assert np.array_equal(a, b)
    assert np.array_equal(a[6], cache[6]) and np.array_equal(a[8], cache[8])


def test_append_image_layouts_are_transposes():
    """The per-block transposed image is the transpose of the row-major one."""
    rng = np.random.default_rng(9)
    cache = rng.integers(0, 65535, size=(10, 3, 4, 5), dtype=np.uint16)
    S = [7, 2, 9]
    P = [0, 8, 4]
    cu = np.concatenate([[0], np.cumsum(S)])
    new = rng.integers(0, 65535, size=(cu[-1], 3, 5), dtype=np.uint16)
    bt = np.array([[0, 1, 2, 9], [3, 4, 5, 9], [6, 7, 8, 9]], dtype=np.int32)
    a = paged.kv_append_image(cache, new, bt, cu, P, 4)
    b = paged.kv_append_image(cache.swapaxes(2, 3), new, bt, cu, P, 4, layout="d_slot")
    assert np.array_equal(a.swapaxes(2, 3), b)


# ---------------------------------------------------------------- out-of-pool table entries
def test_append_image_drops_out_of_pool_writes():
    """A block-table entry outside [0, NB) names no block: its tokens write
    nothing (hand example: entry -1 and entry NB in one row)."""
    cache = np.full((4, 1, 4, 2), 7, dtype=np.uint16)
    new = np.arange(1, 1 + 9 * 2, dtype=np.uint16).reshape(9, 1, 2)
    bt = np.array([[2, -1, 4]], dtype=np.int32)      # tokens 0..3 -> 2, 4..7 dropped, 8 dropped
    for layout, c in (("slot_d", cache), ("d_slot", cache.swapaxes(2, 3).copy())):
        out = paged.kv_append_image(c, new, bt, [0, 9], [0], block_size=4, layout=layout)
        ref = paged.kv_append_image_loops(c, new, bt, [0, 9], [0], block_size=4, layout=layout)
        assert np.array_equal(out, ref)
        blk2 = out[2, 0] if layout == "slot_d" else out[2, 0].T
        assert blk2.tolist() == [[1, 2], [3, 4], [5, 6], [7, 8]]
        for b in (0, 1, 3):                         # untouched, including the last block (-1 must not wrap)
            assert (out[b] == 7).all()


def test_zero_out_of_pool_blocks_hand_example():
    x = np.arange(1, 1 + 11 * 2, dtype=np.float64).reshape(11, 1, 2)   # L = 11, blocks of 4: 3 blocks
    row = np.array([5, -1, 6, 0])                   # NB = 6: block 0 ok, 1 out (-1), 2 out (== NB)
    out = paged.zero_out_of_pool_blocks(x, row, num_blocks=6, block_size=4)
    assert np.array_equal(out[0:4], x[0:4])
    assert (out[4:11] == 0).all()
    out2 = paged.zero_out_of_pool_blocks(x, [0, 1, 2], num_blocks=3, block_size=4)
    assert np.array_equal(out2, x)


def test_out_of_pool_prefix_block_is_a_zero_key_in_the_softmax():
    """Reading of an out-of-pool prefix block: 16 keys of zeros and values of
    zeros, which get weight exp(0) before normalisation. Closed form with the
    other keys' values constant c: O = c * Z_rest / (Z_rest + 16)."""
    rng = np.random.default_rng(3)
    P, S, D, bs = 32, 3, 8, 16
    q = rng.standard_normal((S, 1, D))
    k = rng.standard_normal((P + S, 1, D))
    v = np.full((P + S, 1, D), 2.5)
    kz = paged.zero_out_of_pool_blocks(k, [-1, 0, 1], num_blocks=4, block_size=bs)
    vz = paged.zero_out_of_pool_blocks(v, [-1, 0, 1], num_blocks=4, block_size=bs)
    out = A.suffix_prefill_attention(q, kz, vz, P, 0.5)
    for i in range(S):
        z_rest = np.exp(0.5 * (k[bs:P + i + 1, 0] @ q[i, 0])).sum()
        assert np.allclose(out[i, 0], 2.5 * z_rest / (z_rest + bs), rtol=1e-12, atol=0)
