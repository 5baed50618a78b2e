"""The allocation-free split entry point (cw_suffix_prefill_attn_split_noalloc)
against the split entry point with a caller workspace, through the C ABI:
identical output on two calls in a row, the second with a smaller batch; and
the size limit of its built-in scratch, refused before any device work."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2606_19667_amd import batch as B
from paper_2606_19667_amd import cw
from paper_2606_19667_amd import workload as W


def _say(msg):
    print(msg, flush=True)


def _ragged(hq, hkv, D, S, P, seed):
    prompts = [W.Prompt(uid=i, segments=[(W.SEG_QUESTION_BASE + i, p + s)]) for i, (s, p) in enumerate(zip(S, P))]
    return W.Workload(f"ragged-{hq}q{hkv}kv-d{D}", hq, hkv, D, 16, prompts, seed=seed, prefix_lens=list(P),
                      extra_blocks=5)


def _pair(db, splits):
    """(split path with a caller workspace, allocation-free path) outputs."""
    ref = cw.suffix_prefill_attn_split(db.meta, db.q, db.k_cache, db.v_cache, db.scale, num_splits=splits)
    out = torch.full_like(db.q, 3.0)
    got = cw.suffix_prefill_attn_split_noalloc(db.meta, db.q, db.k_cache, db.v_cache, db.scale,
                                               num_splits=splits, out=out)
    torch.cuda.synchronize()
    assert got.data_ptr() == out.data_ptr()
    return ref, got


@pytest.mark.gpu
def test_noalloc_split_equals_workspace_split_on_two_calls():
    # first call: the question-only batch (16 x 64 rows over 1,344 cached tokens), 2 splits
    w1 = W.question_only()
    _say(f"noalloc first call: {w1.name}")
    db1 = B.materialize(w1, keep_host=[])
    cw.kv_append(db1.meta, db1.k_new, db1.v_new, db1.k_cache, db1.v_cache)
    need1 = cw.split_workspace_bytes(db1.meta, 2)
    assert 0 < need1 <= cw.noalloc_scratch_bytes()
    ref1, got1 = _pair(db1, 2)
    assert torch.equal(ref1.view(torch.int16), got1.view(torch.int16))
    # second call, smaller: a ragged batch with empty and single-row requests, 3 splits
    w2 = _ragged(8, 2, 64, [1, 0, 17, 40], [0, 32, 16, 64], seed=5)
    _say(f"noalloc second call: {w2.name}")
    db2 = B.materialize(w2, keep_host=[])
    cw.kv_append(db2.meta, db2.k_new, db2.v_new, db2.k_cache, db2.v_cache)
    assert cw.split_workspace_bytes(db2.meta, 3) < need1
    ref2, got2 = _pair(db2, 3)
    assert torch.equal(ref2.view(torch.int16), got2.view(torch.int16))
    assert torch.isfinite(got2.float()).all()
    torch.cuda.empty_cache()


def test_noalloc_refuses_batches_beyond_its_scratch():
    """A batch whose partial results exceed the built-in scratch is refused with
    CW_EINVAL before any device call (dummy device pointers are never used)."""
    limit = cw.noalloc_scratch_bytes()
    assert limit == 64 << 20
    hq, hkv, D, splits = 32, 8, 128, 8
    rows = 2000                          # 8 x 2000 x 32 x 128 x 4 bytes > 64 MiB
    cu = np.array([0, rows], np.int32)
    plen = np.array([0], np.int32)
    assert cw.lib().cw_suffix_prefill_split_workspace_bytes(rows, hq, D, splits) > limit
    plan = cw.suffix_prefill_plan(cu, plen, hq, hkv, D, splits)
    d_ = ctypes.c_void_p(16)
    p32 = lambda a: a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    st = cw.lib().cw_suffix_prefill_attn_split_noalloc(d_, d_, d_, d_, 200, d_, d_, p32(cu), p32(plen), 1, hq, hkv,
                                                       D, 16, 1000, 0.1, p32(plan), d_, d_, None)
    assert st == cw.CW_EINVAL
    assert "scratch" in cw.last_error()
