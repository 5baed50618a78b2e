"""GPU parity of libcw's device path against the fp64 CPU oracle.

Every test runs the library's HIP kernels through the C ABI (via the ctypes
binding) on seeded synthetic inputs and compares with the oracle on the same
inputs: bit-exact for the cache image after the append, and for attention
max-abs <= 2e-2 and mean-abs <= 2e-3 against the unrounded fp64 result.
Invariants that hold bitwise for this kernel (prefix cached vs from scratch,
physical placement, batching) are checked bitwise.
"""
import math

import numpy as np
import pytest
import torch

from oracle import attention as OA
from oracle import paged as OP
from paper_2606_19667_amd import batch as B
from paper_2606_19667_amd import cw
from paper_2606_19667_amd import workload as W

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def _say(msg):
    print(msg, flush=True)


def _run(db):
    cw.kv_append(db.meta, db.k_new, db.v_new, db.k_cache, db.v_cache)
    out = cw.suffix_prefill_attn(db.meta, db.q, db.k_cache, db.v_cache, db.scale)
    torch.cuda.synchronize()
    return out


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _check(got, expect, what):
    d = np.abs(got.astype(np.float64) - expect)
    mx, mean = float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0
    _say(f"{what}: max_abs={mx:.3e} mean_abs={mean:.3e} n={d.size}")
    assert np.isfinite(got).all(), what
    assert mx <= MAX_ABS and mean <= MEAN_ABS, (what, mx, mean)


def _compare_full(db, out):
    outs, exps = [], []
    w = db.workload
    for r in range(w.batch):
        c0, c1 = int(db.sched.cu_suffix[r]), int(db.sched.cu_suffix[r + 1])
        P = int(db.sched.prefix_len[r])
        exp = OA.suffix_prefill_attention(db.q_host[r], db.logical_k[r], db.logical_v[r], P, db.scale)
        outs.append(out[c0:c1].float().cpu().numpy())
        exps.append(exp)
    _check(np.concatenate(outs), np.concatenate(exps), w.name)


def _sample_rows(S, rng, n_rows=96):
    """About n_rows distinct suffix rows: the first and last rows, then half
    block-boundary rows (first and last slot of a 16-token block), half uniform."""
    rows = {0, 1, S - 1, S - 2}
    for b in range(0, S, 16):
        rows.update({b, b + 15})
    rows = [x for x in rows if 0 <= x < S]
    rng.shuffle(rows)
    picked = set(int(x) for x in rows[:n_rows // 2]) | {0, S - 1}
    pool = rng.permutation(S)
    for x in pool:
        if len(picked) >= min(n_rows, S):
            break
        picked.add(int(x))
    return sorted(picked)


def _compare_sampled(db, out, requests, seed=0, n_rows=96):
    rng = np.random.default_rng(seed)
    outs, exps = [], []
    for r in requests:
        c0, c1 = int(db.sched.cu_suffix[r]), int(db.sched.cu_suffix[r + 1])
        P = int(db.sched.prefix_len[r])
        rows = _sample_rows(c1 - c0, rng, n_rows)
        exps.append(OA.suffix_prefill_rows(db.q_host[r], db.logical_k[r], db.logical_v[r], P, db.scale, rows))
        outs.append(out[c0:c1][torch.as_tensor(rows, device=out.device)].float().cpu().numpy())
    _check(np.concatenate(outs), np.concatenate(exps), db.workload.name + " (sampled rows)")


def _cleanup():
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


# ------------------------------------------------------------------ append
def _append_check(w):
    db = B.materialize(w, keep_host=[])
    kb, vb = _bits(db.k_cache), _bits(db.v_cache)
    expect_k = OP.kv_append_image(kb, _bits(db.k_new), db.sched.block_table, db.sched.cu_suffix,
                                  db.sched.prefix_len, w.block_size)
    expect_v = OP.kv_append_image(vb, _bits(db.v_new), db.sched.block_table, db.sched.cu_suffix,
                                  db.sched.prefix_len, w.block_size)
    cw.kv_append(db.meta, db.k_new, db.v_new, db.k_cache, db.v_cache)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(db.k_cache), expect_k)
    assert np.array_equal(_bits(db.v_cache), expect_v)
    return db


@pytest.mark.parametrize("make", [W.tiny_single, W.llama8b_single,
                                  lambda: W.llama8b_trace_batch(seed=1, batch=6, warmup=12)])
def test_kv_append_cache_image_is_bit_exact(make):
    w = make()
    _say(f"kv_append {w.name}")
    db = _append_check(w)
    if w.name.startswith("tiny"):
        used = set(db.sched.block_table[0, :6].tolist())
        for b in set(range(8)) - used:           # two unreferenced blocks keep their sentinel
            assert (_bits(db.k_cache)[b] == B.SENTINEL_BITS).all()
            assert (_bits(db.v_cache)[b] == B.SENTINEL_BITS).all()
    _cleanup()


@pytest.mark.parametrize("hq,hkv,D,nreq", [(8, 2, 128, 8), (16, 1, 64, 8), (48, 24, 128, 8),
                                           (40, 20, 64, 8), (8, 8, 128, 70)])
def test_kv_append_ragged_bit_exact(hq, hkv, D, nreq):
    """Partial and empty blocks, head counts that take several staging passes,
    and more requests than one wave scans at a time."""
    if nreq == 8:
        S = [1, 15, 16, 17, 600, 0, 33, 129]
        P = [0, 16, 48, 0, 1024, 32, 1008, 64]
    else:
        rng = np.random.default_rng(nreq)
        S = [int(x) if x % 7 else 0 for x in rng.integers(0, 40, size=nreq)]
        P = [16 * int(x) for x in rng.integers(0, 4, size=nreq)]
    w = _ragged(hq, hkv, D, S, P, seed=hq + D + nreq)
    _say(f"kv_append {w.name} nreq={nreq}")
    _append_check(w)
    _cleanup()


# ------------------------------------------------------------------ attention
def test_attention_tiny_single_request():
    w = W.tiny_single()
    _say(f"attention {w.name}")
    db = B.materialize(w)
    _compare_full(db, _run(db))
    _cleanup()


def test_attention_llama8b_single_request():
    w = W.llama8b_single()
    _say(f"attention {w.name}")
    db = B.materialize(w)
    _compare_full(db, _run(db))
    _cleanup()


def test_attention_small_trace_batch_full():
    w = W.llama8b_trace_batch(seed=2, batch=4, warmup=24)
    _say(f"attention {w.name} P={[None]}")
    db = B.materialize(w)
    _say(f"  prefix_len={db.sched.prefix_len.tolist()}")
    _compare_full(db, _run(db))
    _cleanup()


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_attention_trace_batch16_sampled(seed):
    """The measured 16-request batch at full size; seed 0 is the bench batch."""
    w = W.llama8b_trace_batch(seed=seed)
    _say(f"attention {w.name} seed={seed}")
    db = B.materialize(w)
    _say(f"  prefix_len={db.sched.prefix_len.tolist()}")
    _compare_sampled(db, _run(db), range(w.batch), seed=seed)
    _cleanup()


def test_attention_question_only_full():
    """The short-suffix shape: whole evidence prefix cached, 64-token questions."""
    w = W.question_only()
    _say(f"attention {w.name}")
    db = B.materialize(w)
    _compare_full(db, _run(db))
    _cleanup()


def _ragged(hq, hkv, D, S, P, seed):
    prompts = [W.Prompt(uid=i, segments=[(W.SEG_QUESTION_BASE + i, p + s)]) for i, (s, p) in enumerate(zip(S, P))]
    return W.Workload(f"ragged-{hq}q{hkv}kv-d{D}", hq, hkv, D, 16, prompts, seed=seed, prefix_lens=list(P),
                      extra_blocks=5)


@pytest.mark.parametrize("hq,hkv,D", [(4, 4, 64), (8, 2, 128), (32, 8, 128), (64, 8, 128), (28, 4, 128),
                                      (16, 1, 64), (32, 1, 64), (64, 1, 64), (128, 1, 64), (96, 3, 128)])
def test_attention_ragged_shapes(hq, hkv, D):
    """Ragged lengths (empty, single-row, partial-block and multi-tile suffixes)
    at every tile shape: G = Hq / Hkv query heads share a tile of 256 / G
    positions, from 256 positions (G = 1) down to 2 (G = 128)."""
    S = [1, 15, 16, 17, 600, 0, 33, 129]
    P = [0, 16, 48, 0, 1024, 32, 1008, 64]
    w = _ragged(hq, hkv, D, S, P, seed=hq + D)
    _say(f"attention {w.name} S={S} P={P}")
    db = B.materialize(w)
    _compare_full(db, _run(db))
    _cleanup()


# ------------------------------------------------------------------ invariants (bitwise)
def test_prefix_cached_equals_full_prefill_bitwise():
    """Rows P.. of a from-scratch prefill of all L tokens equal the prefill of the
    suffix over the cached prefix, bit for bit (tiles are anchored to absolute
    key positions and fully masked tiles leave a row's state unchanged)."""
    base = W.llama8b_single()
    full = W.Workload("llama8b-single-p0", 32, 8, 128, 16, base.prompts, seed=0, prefix_lens=[0])
    a = B.materialize(base)
    out_a = _run(a)
    b = B.materialize(full, keep_host=[])
    out_b = _run(b)
    assert torch.equal(out_a.view(torch.int16), out_b[832:].view(torch.int16))
    _cleanup()


def test_physical_placement_does_not_change_output():
    w1 = W.llama8b_single()
    w2 = W.llama8b_single()
    w2.free_order_key = (99,)
    assert not np.array_equal(w1.free_order(), w2.free_order())
    o1 = _run(B.materialize(w1, keep_host=[]))
    o2 = _run(B.materialize(w2, keep_host=[]))
    assert torch.equal(o1.view(torch.int16), o2.view(torch.int16))
    _cleanup()


def test_request_alone_equals_request_in_batch():
    w = W.llama8b_trace_batch(seed=3, batch=5, warmup=16)
    db = B.materialize(w, keep_host=[])
    out = _run(db)
    r = 3
    single = W.Workload("alone", 32, 8, 128, 16, [w.prompts[r]], seed=w.seed, content="blocks",
                        prefix_lens=[int(db.sched.prefix_len[r])])
    o1 = _run(B.materialize(single, keep_host=[]))
    c0, c1 = int(db.sched.cu_suffix[r]), int(db.sched.cu_suffix[r + 1])
    assert torch.equal(out[c0:c1].view(torch.int16), o1.view(torch.int16))
    _cleanup()


# ------------------------------------------------------------------ full-size shapes, sampled rows
@pytest.mark.parametrize("frac", [0.0, 0.3, 0.6, 0.9])
def test_topk_sweep_sampled(frac):
    w = W.topk_sweep(frac)
    _say(f"attention {w.name}")
    db = B.materialize(w, keep_host=[0, w.batch - 1], gen_device="cuda")
    _compare_sampled(db, _run(db), [0, w.batch - 1])
    del db
    _cleanup()


@pytest.mark.parametrize("hit", ["low", "high"])
def test_long_context_70b_sampled(hit):
    """Two requests x all 64 heads x 256 sampled rows each (first and last rows,
    block boundaries, uniform rows)."""
    w = W.long_context(hit)
    _say(f"attention {w.name} P={w.prefix_lens[:4]}...")
    db = B.materialize(w, keep_host=[0, w.batch - 1], gen_device="cuda")
    _compare_sampled(db, _run(db), [0, w.batch - 1], n_rows=256)
    del db
    _cleanup()


def test_prebound_runner_matches_binding_path_bitwise():
    """The pre-bound path the bench times (one schedule call, one packed upload,
    cached launch arguments) computes exactly what the plain binding computes."""
    w = W.llama8b_trace_batch(seed=4, batch=6, warmup=20)
    db = B.materialize(w, keep_host=[])
    ref = _run(db)
    stride = B.bt_stride_for(w)
    pool = cw.Pool(w.num_blocks(), w.free_order())
    for p in w.warmup:
        bt, pl, cu = cw.schedule_batch(pool, [p.tokens(w.seed)], stride)
        cw.release_batch(pool, bt, pl, cu)
    rn = cw.BatchRunner([p.tokens(w.seed) for p in w.prompts], stride, w.num_q_heads, w.num_kv_heads,
                        w.head_dim)
    rn.schedule(pool)
    assert np.array_equal(rn.bt_host, db.sched.block_table) and np.array_equal(rn.plen_host, db.sched.prefix_len)
    out = torch.empty_like(db.q)
    k2, v2 = db.k_cache.clone(), db.v_cache.clone()
    rn.bind(db.q, db.k_new, db.v_new, k2, v2, out, w.scale)
    rn.upload()
    rn.kv_append()
    rn.attention()
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    assert torch.equal(k2.view(torch.int16), db.k_cache.view(torch.int16))
    rn.release(pool)
    _cleanup()


# ------------------------------------------------------------------ out-of-pool table entries
def _with_table(db, bt):
    """The batch with another block table (host and device copies)."""
    w = db.workload
    db.sched.block_table = bt
    db.meta = cw.BatchMeta(bt, db.sched.cu_suffix, db.sched.prefix_len, w.num_q_heads, w.num_kv_heads,
                           w.head_dim, db.q.device)
    return db


def _corrupt_table(db):
    """Entries -1, num_blocks and num_blocks + 7 inside requests' prompts:
    prefix blocks of request 1 and 2, a suffix block of request 2."""
    bt = db.sched.block_table.copy()
    nb = db.sched.num_blocks
    bt[1, 1] = -1
    bt[1, 3] = nb
    bt[2, 0] = nb + 7
    P2 = int(db.sched.prefix_len[2])
    bt[2, P2 // 16 + 1] = -1                      # a suffix block: its append is dropped
    return bt


def _oop_workload():
    S = [40, 70, 100]
    P = [32, 64, 96]
    return _ragged(8, 2, 128, S, P, seed=77)


def test_kv_append_drops_out_of_pool_writes_bit_exact():
    w = _oop_workload()
    db = B.materialize(w, keep_host=[])
    db = _with_table(db, _corrupt_table(db))
    _say(f"kv_append out-of-pool entries {w.name}")
    kb, vb = _bits(db.k_cache), _bits(db.v_cache)
    expect_k = OP.kv_append_image(kb, _bits(db.k_new), db.sched.block_table, db.sched.cu_suffix,
                                  db.sched.prefix_len, w.block_size)
    expect_v = OP.kv_append_image(vb, _bits(db.v_new), db.sched.block_table, db.sched.cu_suffix,
                                  db.sched.prefix_len, w.block_size)
    cw.kv_append(db.meta, db.k_new, db.v_new, db.k_cache, db.v_cache)
    torch.cuda.synchronize()
    assert np.array_equal(_bits(db.k_cache), expect_k)
    assert np.array_equal(_bits(db.v_cache), expect_v)
    _cleanup()


def test_attention_reads_out_of_pool_blocks_as_zeros():
    """Against the oracle with the logical K/V rows of every out-of-pool block
    of a request zeroed (prefix and suffix blocks alike)."""
    w = _oop_workload()
    db = B.materialize(w)
    db = _with_table(db, _corrupt_table(db))
    _say(f"attention out-of-pool entries {w.name}")
    out = _run(db)
    nb = db.sched.num_blocks
    outs, exps = [], []
    for r in range(w.batch):
        c0, c1 = int(db.sched.cu_suffix[r]), int(db.sched.cu_suffix[r + 1])
        P = int(db.sched.prefix_len[r])
        row = db.sched.block_table[r]
        k = OP.zero_out_of_pool_blocks(db.logical_k[r], row, nb)
        v = OP.zero_out_of_pool_blocks(db.logical_v[r], row, nb)
        exps.append(OA.suffix_prefill_attention(db.q_host[r], k, v, P, db.scale))
        outs.append(out[c0:c1].float().cpu().numpy())
    _check(np.concatenate(outs), np.concatenate(exps), w.name + " (out-of-pool entries)")
    _cleanup()


# ------------------------------------------------------------------ plan binding on the device
def test_device_plan_of_another_batch_computes_nothing():
    """A device plan whose header fingerprint is not the validated batch's: the
    kernel writes nothing (the host copy passed validation)."""
    w = W.tiny_single()
    db = B.materialize(w, keep_host=[])
    cw.kv_append(db.meta, db.k_new, db.v_new, db.k_cache, db.v_cache)
    db.meta.plan[2] += 1                        # fingerprint word of the device copy only
    sentinel = torch.full_like(db.q, 7.0)
    cw.suffix_prefill_attn(db.meta, db.q, db.k_cache, db.v_cache, db.scale, out=sentinel)
    torch.cuda.synchronize()
    assert torch.all(sentinel == 7.0)
    db.meta.plan[2] -= 1
    cw.suffix_prefill_attn(db.meta, db.q, db.k_cache, db.v_cache, db.scale, out=sentinel)
    torch.cuda.synchronize()
    assert not torch.all(sentinel == 7.0)
    _cleanup()
