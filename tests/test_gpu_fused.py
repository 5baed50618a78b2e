"""GPU parity of the fused append + attention call (cw_suffix_prefill_append_attn).

The fused call must leave the caches and write the output exactly as
cw_kv_append followed by cw_suffix_prefill_attn does on the same inputs: both
are compared bit for bit with that sequence, the cache image also with the
oracle's append image, and the output with the fp64 oracle (max-abs <= 2e-2,
mean-abs <= 2e-3), in full for small batches and on sampled rows for large ones.
"""
import numpy as np
import pytest
import torch

import test_gpu_parity as GP
from oracle import paged as OP
from paper_2606_19667_amd import batch as B
from paper_2606_19667_amd import cw
from paper_2606_19667_amd import workload as W

pytestmark = pytest.mark.gpu


def _fused(db):
    out = cw.suffix_prefill_append_attn(db.meta, db.q, db.k_new, db.v_new, db.k_cache, db.v_cache, db.scale)
    torch.cuda.synchronize()
    return out


def _pair(w, table=None, keep_host=None, gen_device=None):
    """Two copies of the batch (the same seeded inputs), optionally with
    another block table: the sequential calls run on the first, the fused call
    on the second. Returns both batches, both outputs and the oracle's append
    image of the second's caches."""
    dbs = []
    for _ in range(2):
        db = B.materialize(w, keep_host=keep_host, gen_device=gen_device)
        if table is not None:
            db = GP._with_table(db, table(db))
        dbs.append(db)
    seq, fus = dbs
    img = []
    for cache, new in ((fus.k_cache, fus.k_new), (fus.v_cache, fus.v_new)):
        img.append(OP.kv_append_image(GP._bits(cache), GP._bits(new), fus.sched.block_table, fus.sched.cu_suffix,
                                      fus.sched.prefix_len, w.block_size))
    out_s = GP._run(seq)
    out_f = _fused(fus)
    return seq, fus, out_s, out_f, img


def _check_same(seq, fus, out_s, out_f, img, what):
    GP._say(f"fused vs sequential {what}: rows={int(fus.sched.cu_suffix[-1])}")
    assert torch.equal(out_f.view(torch.int16), out_s.view(torch.int16)), what + ": output"
    assert torch.equal(fus.k_cache.view(torch.int16), seq.k_cache.view(torch.int16)), what + ": K cache"
    assert torch.equal(fus.v_cache.view(torch.int16), seq.v_cache.view(torch.int16)), what + ": V cache"
    assert np.array_equal(GP._bits(fus.k_cache), img[0]), what + ": K cache vs oracle image"
    assert np.array_equal(GP._bits(fus.v_cache), img[1]), what + ": V cache vs oracle image"


@pytest.mark.parametrize("make", [W.tiny_single, W.llama8b_single, W.question_only,
                                  lambda: W.llama8b_trace_batch(seed=2, batch=4, warmup=24)])
def test_fused_small_batches_full(make):
    w = make()
    GP._say(f"fused {w.name}")
    seq, fus, out_s, out_f, img = _pair(w)
    _check_same(seq, fus, out_s, out_f, img, w.name)
    GP._compare_full(fus, out_f)
    GP._cleanup()


def test_fused_trace_batch16_reads_same_batch_blocks_from_new_rows():
    """The measured 16-request batch: some requests' prefix blocks are blocks
    an earlier request of the batch commits in the same schedule."""
    w = W.llama8b_trace_batch(seed=0)
    GP._say(f"fused {w.name}")
    seq, fus, out_s, out_f, img = _pair(w)
    t = cw.append_table(fus.meta.append_plan(fus.sched.num_blocks)[0])
    pending = sum(int(((t[r, :int(fus.sched.prefix_len[r]) // 16, 0] < 0) &
                       (t[r, :int(fus.sched.prefix_len[r]) // 16, 0] != -1)).sum()) for r in range(w.batch))
    GP._say(f"  prefix blocks of the same batch: {pending}")
    assert pending > 0
    _check_same(seq, fus, out_s, out_f, img, w.name)
    GP._compare_sampled(fus, out_f, range(w.batch))
    GP._cleanup()


@pytest.mark.parametrize("hq,hkv,D", [(4, 4, 64), (8, 2, 128), (32, 8, 128), (64, 8, 128), (28, 4, 128),
                                      (16, 1, 64), (32, 1, 64), (128, 1, 64), (96, 3, 128)])
def test_fused_ragged_shapes(hq, hkv, D):
    """Empty, single-row, partial-block and multi-tile suffixes at tile shapes
    from 256 positions per tile (G = 1) down to 2 (G = 128): an entry's own
    rows span several blocks, one block, or part of one."""
    S = [1, 15, 16, 17, 600, 0, 33, 129]
    P = [0, 16, 48, 0, 1024, 32, 1008, 64]
    w = GP._ragged(hq, hkv, D, S, P, seed=hq + D)
    GP._say(f"fused {w.name}")
    seq, fus, out_s, out_f, img = _pair(w)
    _check_same(seq, fus, out_s, out_f, img, w.name)
    GP._compare_full(fus, out_f)
    GP._cleanup()


def test_fused_out_of_pool_entries():
    """Table entries -1 and >= num_blocks in prefix and suffix blocks: writes
    dropped, reads as zeros, as in the two calls."""
    w = GP._oop_workload()
    GP._say(f"fused out-of-pool entries {w.name}")
    seq, fus, out_s, out_f, img = _pair(w, table=GP._corrupt_table, keep_host=[])
    _check_same(seq, fus, out_s, out_f, img, w.name + " (out-of-pool entries)")
    GP._cleanup()


def test_fused_prefix_blocks_that_are_suffix_blocks_of_the_batch():
    """A hand-made table in which request 1's prefix blocks are full suffix
    blocks of request 0 and request 2's prefix block is one of request 1's:
    they hold the appended rows, which the fused call reads from k_new / v_new."""
    S, P = [48, 20, 40], [0, 32, 16]
    w = GP._ragged(8, 2, 128, S, P, seed=5)

    def alias(db):
        bt = db.sched.block_table.copy()
        bt[1, 0], bt[1, 1] = bt[0, 2], bt[0, 1]
        bt[2, 0] = bt[1, 2]          # request 1's first suffix block (rows 0..15, full)
        return bt
    seq, fus, out_s, out_f, img = _pair(w, table=alias, keep_host=[])
    t = cw.append_table(fus.meta.append_plan(fus.sched.num_blocks)[0])
    rows = lambda R: int(np.array([0x80000000 | R], np.uint32).view(np.int32)[0])   # noqa: E731
    assert t[1, 0, 0] == rows(32) and t[1, 1, 0] == rows(16) and t[2, 0, 0] == rows(48)
    _check_same(seq, fus, out_s, out_f, img, w.name + " (same-batch prefix blocks)")
    GP._cleanup()


@pytest.mark.parametrize("hit", ["high"])
def test_fused_long_context_70b_sampled(hit):
    w = W.long_context(hit)
    GP._say(f"fused {w.name}")
    seq, fus, out_s, out_f, img = _pair(w, keep_host=[0, w.batch - 1], gen_device="cuda")
    _check_same(seq, fus, out_s, out_f, img, w.name)
    GP._compare_sampled(fus, out_f, [0, w.batch - 1], n_rows=128)
    del seq, fus
    GP._cleanup()


def test_fused_runner_matches_sequential_calls_bitwise():
    """The pre-bound fused path the bench times (schedule with the fused plan,
    one packed upload, cached launch arguments)."""
    w = W.llama8b_trace_batch(seed=4, batch=6, warmup=20)
    db = B.materialize(w, keep_host=[])
    k0, v0 = db.k_cache.clone(), db.v_cache.clone()
    ref = GP._run(db)
    stride = B.bt_stride_for(w)
    pool = cw.Pool(w.num_blocks(), w.free_order())
    for p in w.warmup:
        bt, pl, cu = cw.schedule_batch(pool, [p.tokens(w.seed)], stride)
        cw.release_batch(pool, bt, pl, cu)
    rn = cw.BatchRunner([p.tokens(w.seed) for p in w.prompts], stride, w.num_q_heads, w.num_kv_heads,
                        w.head_dim, fused=True)
    out = torch.empty_like(db.q)
    rn.bind(db.q, db.k_new, db.v_new, k0, v0, out, w.scale)
    rn.schedule(pool)
    assert np.array_equal(rn.bt_host, db.sched.block_table)
    rn.upload()
    rn.append_attention()
    torch.cuda.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))
    assert torch.equal(k0.view(torch.int16), db.k_cache.view(torch.int16))
    assert torch.equal(v0.view(torch.int16), db.v_cache.view(torch.int16))
    rn.release(pool)
    GP._cleanup()
