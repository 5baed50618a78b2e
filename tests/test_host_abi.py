"""Host side of libcw on the CPU: exported symbols, hashes, the block pool,
batch scheduling, the tile planner and argument validation of the device entry
points (which fail before touching a GPU). Expected values come from the
oracle package."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

from oracle import paged
from paper_2606_19667_amd import cw, workload as W

HEADER = os.path.join(os.path.dirname(os.path.dirname(__file__)), "include", "cw.h")


def test_exports_every_declared_symbol():
    text = open(HEADER).read()
    declared = set(re.findall(r"\b(cw_[a-z0-9_]+)\s*\(", text))
    assert declared == set(cw.EXPORTED)
    lib = ctypes.CDLL(cw.LIB_PATH)
    for name in declared:
        assert hasattr(lib, name), name
    assert cw.abi_version() == 4


@pytest.mark.parametrize("n", [0, 1, 15, 16, 17, 100, 1408])
def test_block_hashes_match_oracle(n):
    toks = np.random.default_rng(n).integers(-2**31, 2**31 - 1, size=n, dtype=np.int64).astype(np.int32)
    got = cw.block_hashes(toks, 16)
    assert [int(x) for x in got] == paged.chain_block_hashes(toks, 16)


def test_block_hashes_other_block_sizes():
    toks = np.arange(100, dtype=np.int32)
    for bs in (1, 7, 32):
        assert [int(x) for x in cw.block_hashes(toks, bs)] == paged.chain_block_hashes(toks, bs)


def _same_error(fn_a, fn_b):
    ea = eb = None
    ra = rb = None
    try:
        ra = fn_a()
    except cw.CwError as e:
        ea = e.status
    try:
        rb = fn_b()
    except ValueError:
        eb = "err"
    assert (ea is None) == (eb is None), (ea, eb)
    return ra, rb


def test_pool_matches_oracle_on_random_operations():
    rng = np.random.default_rng(11)
    for trial in range(20):
        nb = int(rng.integers(4, 40))
        order = rng.permutation(nb)
        c = cw.Pool(nb, order)
        o = paged.PoolSim(nb, order)
        hash_space = [int(x) for x in rng.integers(1, 2**63, size=12)]
        held = []
        for step in range(300):
            op = rng.integers(0, 4)
            if op == 0:
                n = int(rng.integers(0, 6))
                a, b = _same_error(lambda: c.alloc(n), lambda: o.alloc(n))
                if a is not None:
                    assert a.tolist() == b
                    held += b
            elif op == 1:
                hs = [hash_space[int(i)] for i in rng.integers(0, len(hash_space), size=int(rng.integers(0, 5)))]
                cap = int(rng.integers(0, 6))
                a = c.prefix_match(hs, cap)
                b = o.prefix_match(hs, cap)
                assert a.tolist() == b
                held += b
            elif op == 2 and held:
                k = int(rng.integers(1, min(4, len(held)) + 1))
                ids = [held[int(i)] for i in rng.choice(len(held), size=k, replace=False)]
                if rng.random() < 0.1:
                    ids = ids + [int(rng.integers(0, nb))]
                hs = [hash_space[int(i)] for i in rng.integers(0, len(hash_space), size=len(ids))]
                _same_error(lambda: c.commit(hs, ids), lambda: o.commit(hs, ids))
            elif op == 3 and held:
                k = int(rng.integers(1, min(4, len(held)) + 1))
                idx = sorted(rng.choice(len(held), size=k, replace=False).tolist(), reverse=True)
                ids = [held[i] for i in idx]
                if rng.random() < 0.1:
                    ids = ids + [int(rng.integers(0, nb))]
                a, b = _same_error(lambda: c.release(ids), lambda: o.release(ids))
                if a is None and b is None and not isinstance(a, Exception):
                    pass
                if o.ref == [int(x) for x in o.ref]:
                    pass
                # keep `held` in sync with the oracle's counts
                held = [b2 for b2 in range(nb) for _ in range(o.ref[b2])]
            assert c.num_free == len(o.free)
        # the free-queue order decides future allocations
        assert c.alloc(c.num_free).tolist() == o.alloc(len(o.free))


def _simulate_oracle(prompts, pool, bs, stride):
    tables, plens, cus = [], [], [0]
    for toks in prompts:
        hs = paged.chain_block_hashes(toks, bs)
        ids = pool.prefix_match(hs, (len(toks) - 1) // bs)
        new = pool.alloc(math.ceil(len(toks) / bs) - len(ids))
        pool.commit(hs[len(ids):], new[:len(hs) - len(ids)])
        row = ids + new
        tables.append(row + [-1] * (stride - len(row)))
        plens.append(len(ids) * bs)
        cus.append(cus[-1] + len(toks) - len(ids) * bs)
    return np.array(tables, np.int32), np.array(plens, np.int32), np.array(cus, np.int32)


def test_schedule_batch_matches_oracle_on_trace():
    w = W.llama8b_trace_batch(seed=0, batch=16, warmup=48)
    prompts = [p.tokens(w.seed) for p in w.warmup + w.prompts]
    nb = w.num_blocks()
    order = w.free_order()
    c = cw.Pool(nb, order)
    o = paged.PoolSim(nb, order)
    stride = 88
    for toks in prompts[:len(w.warmup)]:
        bt, pl, cu = cw.schedule_batch(c, [toks], stride)
        ebt, epl, ecu = _simulate_oracle([toks], o, 16, stride)
        assert np.array_equal(bt, ebt) and np.array_equal(pl, epl) and np.array_equal(cu, ecu)
        cw.release_batch(c, bt, pl, cu)
        o.release([b for b in ebt[0] if b >= 0])
    batch = prompts[len(w.warmup):]
    bt, pl, cu = cw.schedule_batch(c, batch, stride)
    ebt, epl, ecu = _simulate_oracle(batch, o, 16, stride)
    assert np.array_equal(bt, ebt) and np.array_equal(pl, epl) and np.array_equal(cu, ecu)
    # depths are whole documents past the instruction; the greedy depth is a lower bound
    for p, d in zip(pl, w.trie_depths):
        assert (p - 64) % 256 == 0 and p >= 64 + 256 * d
    cw.release_batch(c, bt, pl, cu)


def test_schedule_batch_rolls_back_on_exhaustion():
    c = cw.Pool(10)
    a = c.alloc(3)
    c.commit([1, 2, 3], a)
    c.release(a)
    snap = c.clone()
    prompts = [np.arange(48, dtype=np.int32), np.arange(1000, 1000 + 16 * 9, dtype=np.int32)]
    with pytest.raises(cw.CwError) as e:
        cw.schedule_batch(c, prompts, 16)
    assert e.value.status == cw.CW_ENOSPC
    assert c.num_free == snap.num_free == 10
    assert c.alloc(10).tolist() == snap.alloc(10).tolist()


def test_schedule_batch_keeps_one_suffix_token_and_shares_within_batch():
    c = cw.Pool(64)
    p = np.arange(64, dtype=np.int32)
    bt, pl, cu = cw.schedule_batch(c, [p, p, np.concatenate([p, [7]])], 8)
    assert pl.tolist() == [0, 48, 64]          # cap (L-1)//16 blocks; same-batch reuse
    assert cu.tolist() == [0, 64, 80, 81]
    assert bt[1, :3].tolist() == bt[0, :3].tolist() and bt[2, :4].tolist() == bt[0, :4].tolist()
    assert bt[0, 4:].tolist() == [-1] * 4


def _entries(plan):
    """Real entries of a plan with their queue (workgroup) and queue position."""
    grid, qlen = int(plan[cw.HDR_GRID]), int(plan[cw.HDR_QUEUE_LEN])
    ents = cw.plan_entries(plan)
    assert len(ents) == grid * qlen == plan[cw.HDR_ENTRIES]
    out = []
    for w in range(grid):
        ended = False
        for i in range(qlen):
            e = ents[i * grid + w]
            if e[cw.ENT_R] < 0:
                ended = True
                continue
            assert not ended, "a real entry after the end of its queue"
            out.append((w, i, e))
    return out


def _check_plan(plan, cu, P, hq, hkv, splits=1):
    """Every (request, KV head, row) is covered by exactly one tile, and each
    tile's 64-key steps by its split runs exactly once, in order; the fields
    are the batch's own."""
    per = cw.TILE_ROWS // (hq // hkv)
    rows, runs = {}, {}
    for w, i, e in _entries(plan):
        r, g, row0, nv, cu0, p, L, kb, ke, sp = (int(x) for x in e[:10])
        S = cu[r + 1] - cu[r]
        assert 0 <= g < hkv and row0 % per == 0 and nv == min(per, S - row0) and nv >= 1
        assert cu0 == cu[r] and p == P[r] and L == P[r] + S
        n = -(-(p + row0 + nv) // 64)
        assert 0 <= sp < splits and kb == n * sp // splits and ke == n * (sp + 1) // splits
        runs.setdefault((r, g, row0), []).append((sp, kb, ke, n))
        if sp == 0:
            for row in range(row0, row0 + nv):
                rows[(r, g, row)] = rows.get((r, g, row), 0) + 1
    assert len(rows) == int(np.sum(np.diff(cu))) * hkv and set(rows.values()) <= {1}
    for key, rr in runs.items():
        rr.sort()
        assert [x[0] for x in rr] == list(range(splits))
        n = rr[0][3]
        steps = [t for _, kb, ke, _ in rr for t in range(kb, ke)]
        assert steps == list(range(n))
    return per


def _grouped(plan):
    """True when each (request, KV head) pair's entries sit on one partition (queue % 8)."""
    part = {}
    for w, i, e in _entries(plan):
        if part.setdefault((int(e[0]), int(e[1])), w % 8) != w % 8:
            return False
    return len(part) >= 32


@pytest.mark.parametrize("shape", [(4, 1), (32, 8), (64, 8), (28, 4), (128, 1)])
def test_plan_covers_every_row_and_step_once(shape):
    hq, hkv = shape
    rng = np.random.default_rng(hq)
    for B in (1, 3, 16, 40):
        S = rng.integers(0, 700, size=B)
        S[0] = max(S[0], 1)
        P = rng.integers(0, 60, size=B) * 16
        cu = np.concatenate([[0], np.cumsum(S)]).astype(np.int32)
        for splits in (1, 3):
            plan = cw.suffix_prefill_plan(cu, P, hq, hkv, 128, splits)
            assert plan[0] == 0x33505743 and plan[cw.HDR_SPLITS] == splits
            per = _check_plan(plan, cu, P, hq, hkv, splits)
            ents = _entries(plan)
            assert len(ents) == sum(math.ceil(s / per) for s in S) * hkv * splits
            assert plan[cw.HDR_GRID] == min(256, len(ents))


def _queue_loads(plan):
    load, heavy = {}, 0
    for w, i, e in _entries(plan):
        c = int(e[cw.ENT_KEND] - e[cw.ENT_KBEG]) + 1
        load[w] = load.get(w, 0) + c
        heavy = max(heavy, c)
    return load, heavy


def test_plan_queues_are_balanced_longest_first():
    """Without partition grouping (fewer than 32 pairs), each queue runs its
    entries heaviest first, and no queue carries more than the lightest queue
    plus its heaviest entry (list scheduling)."""
    rng = np.random.default_rng(5)
    S = rng.integers(1, 1400, size=3)
    P = rng.integers(0, 20, size=3) * 64
    cu = np.concatenate([[0], np.cumsum(S)]).astype(np.int32)
    plan = cw.suffix_prefill_plan(cu, P, 32, 8, 128)
    assert not _grouped(plan)
    last = {}
    for w, i, e in _entries(plan):
        c = int(e[cw.ENT_KEND] - e[cw.ENT_KBEG]) + 1
        assert c <= last.get(w, 1 << 30)
        last[w] = c
    load, heavy = _queue_loads(plan)
    assert max(load.values()) <= min(load.values()) + heavy


@pytest.mark.parametrize("splits", [6, 8, 16])
def test_split_plan_spreads_empty_runs(splits):
    """A single request with tiles of fewer steps than splits (some runs are
    empty): the runs of a tile differ by at most one step, and the queues stay
    balanced with an empty run counted as one step (regression: at cost 0
    every empty run landed on one queue, 66 entries deep at 8 splits)."""
    cu = np.array([0, 576], np.int32)
    P = np.array([832], np.int32)
    plan = cw.suffix_prefill_plan(cu, P, 32, 8, 128, splits)
    _check_plan(plan, cu, P, 32, 8, splits)
    per_tile = {}
    for w, i, e in _entries(plan):
        per_tile.setdefault((int(e[0]), int(e[1]), int(e[2])), []).append(int(e[cw.ENT_KEND] - e[cw.ENT_KBEG]))
    for steps in per_tile.values():
        assert max(steps) - min(steps) <= 1
    n_entries = len(_entries(plan))
    grid = int(plan[cw.HDR_GRID])
    assert int(plan[cw.HDR_QUEUE_LEN]) <= -(-n_entries // grid) + 1
    load, heavy = _queue_loads(plan)
    assert max(load.values()) <= min(load.values()) + heavy


def test_grouped_plan_runs_rounds_in_pair_order_and_stays_balanced():
    """With partition grouping, the entries a partition's queues hold at one
    queue position (a round, run at about the same time) are consecutive in
    (pair, split run, first row) order, rounds follow each other in that
    order, and the queues stay balanced within one entry's work."""
    rng = np.random.default_rng(5)
    S = rng.integers(1, 1400, size=16)
    P = rng.integers(0, 20, size=16) * 64
    cu = np.concatenate([[0], np.cumsum(S)]).astype(np.int32)
    for hkv, splits in ((8, 1), (4, 1), (8, 2)):
        plan = cw.suffix_prefill_plan(cu, P, 32, hkv, 128, splits)
        assert _grouped(plan)
        qlen = int(plan[cw.HDR_QUEUE_LEN])
        for x in range(8):
            rounds = []
            for i in range(qlen):
                keys = sorted((int(e[0]) * hkv + int(e[1]), int(e[cw.ENT_SPLIT]), int(e[cw.ENT_ROW0]))
                              for w, j, e in _entries(plan) if w % 8 == x and j == i)
                if keys:
                    rounds.append(keys)
            # all but the last three rounds (placed longest first) are runs of
            # the sorted order, one after another
            body = rounds[:-3]
            flat = [k for r in body for k in r]
            assert flat == sorted(flat)
            assert all(len(r) == 32 for r in body)
        load, heavy = _queue_loads(plan)
        assert max(load.values()) <= min(load.values()) + heavy


@pytest.mark.parametrize("grouped", [False, True])
def test_plan_writes_exactly_plan_words(grouped):
    """The plan fills exactly the size cw_suffix_prefill_plan_words reports, with
    empty requests anywhere in the batch (guard words after the buffer stay
    intact); a smaller buffer is refused."""
    B = 40 if grouped else 3
    S = np.array([0, 5, 0, 700, 33, 0] * 7, dtype=np.int32)[:B]
    P = np.arange(B, dtype=np.int32) % 5 * 16
    cu = np.concatenate([[0], np.cumsum(S)]).astype(np.int32)
    cu_a, cu_p = _arr(cu)
    pl_a, pl_p = _arr(P)
    words = cw.lib().cw_suffix_prefill_plan_words(cu_p, pl_p, B, 32, 8, 128, 1)
    assert words > 16
    buf = np.full(words + 256, -7, dtype=np.int32)
    bp = buf.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    assert cw.lib().cw_suffix_prefill_plan(cu_p, pl_p, B, 32, 8, 128, 1, bp, words - 1) == cw.CW_EINVAL
    assert cw.lib().cw_suffix_prefill_plan(cu_p, pl_p, B, 32, 8, 128, 1, bp, words) == cw.CW_OK
    assert words == 16 + 16 * buf[cw.HDR_ENTRIES]
    assert (buf[words:] == -7).all()
    assert _grouped(buf[:words]) == grouped
    _check_plan(buf[:words], cu, P, 32, 8)


def test_plan_groups_pairs_on_one_partition():
    cu = np.arange(0, 17 * 576, 576, dtype=np.int32)
    P = np.full(16, 832, np.int32)
    assert _grouped(cw.suffix_prefill_plan(cu, P, 32, 8, 128))


def test_plan_check_words_bind_entries_to_the_batch():
    """Each entry's check word derives from the batch fingerprint and the
    entry's position: plans of two batches that differ in one prefix length
    differ in every real entry's check word."""
    cu = np.array([0, 300, 900], np.int32)
    a = cw.suffix_prefill_plan(cu, [0, 64], 32, 8, 128)
    b = cw.suffix_prefill_plan(cu, [0, 80], 32, 8, 128)
    assert tuple(a[2:4]) != tuple(b[2:4])
    ea, eb = cw.plan_entries(a), cw.plan_entries(b)
    real = ea[:, 0] >= 0
    assert (ea[real, 15] != eb[real, 15]).all()


def _dummy():
    return ctypes.c_void_p(16)


def _arr(x):
    a = np.ascontiguousarray(x, np.int32)
    return a, a.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))


def _attn(cu, plen, hq=32, hkv=8, d=128, bs=16, stride=100, scale=0.1, nb=100, plan=None, split=False,
          ws_bytes=None, workspace=True):
    """Calls an attention entry point with dummy device pointers (never
    dereferenced: every case here returns before a launch)."""
    cu_a, cu_p = _arr(cu)
    pl_a, pl_p = _arr(plen)
    if plan is None:
        try:
            plan = cw.suffix_prefill_plan(cu, plen, hq, hkv, d)
        except cw.CwError:
            plan = np.zeros(16, np.int32)
    plan = np.ascontiguousarray(plan, np.int32)
    pp = plan.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    d_ = _dummy()
    if not split:
        return cw.lib().cw_suffix_prefill_attn(d_, d_, d_, d_, stride, d_, d_, cu_p, pl_p, len(plen), hq, hkv, d,
                                               bs, nb, scale, pp, d_, d_, None)
    if ws_bytes is None:
        ws_bytes = max(0, cw.lib().cw_suffix_prefill_split_workspace_bytes(cu[-1], hq, d, int(max(1, plan[5]))))
    return cw.lib().cw_suffix_prefill_attn_split(d_, d_, d_, d_, stride, d_, d_, cu_p, pl_p, len(plen), hq, hkv, d,
                                                 bs, nb, scale, pp, d_, d_ if workspace else None, ws_bytes, d_, None)


def _append(cu, plen, hkv=8, d=128, bs=16, stride=100, nb=100):
    cu_a, cu_p = _arr(cu)
    pl_a, pl_p = _arr(plen)
    d_ = _dummy()
    return cw.lib().cw_kv_append(d_, d_, d_, d_, d_, stride, d_, d_, cu_p, pl_p, len(plen), hkv, d, bs, nb, None)


def test_device_entry_points_validate_before_launch():
    E, U = cw.CW_EINVAL, cw.CW_EUNSUPPORTED
    assert _attn([0, 10], [8]) == E                       # prefix not a multiple of 16
    assert _attn([0, 10, 5], [0, 0]) == E                 # cu decreasing
    assert _attn([1, 10], [0]) == E                       # cu[0] != 0
    assert _attn([0, 1000], [16 * 90]) == E               # needs more blocks than the stride
    assert _attn([0, 10], [0], hq=30, hkv=8) == E         # Hq % Hkv
    assert _attn([0, 10], [0], d=96) == U                 # head_dim
    assert _attn([0, 10], [0], bs=32) == U                # block size
    assert _attn([0, 10], [0], hq=256, hkv=1) == U        # group > 128
    other = cw.suffix_prefill_plan([0, 10], [16], 32, 8, 128)
    assert _attn([0, 10], [0], plan=other) == E           # a plan of another batch
    assert "another batch" in cw.last_error()
    assert _attn([0, 10], [0], plan=cw.suffix_prefill_plan([0, 10], [0], 16, 4, 128)) == E   # other heads
    assert _attn([0, 10], [0], plan=np.zeros(16, np.int32)) == E      # not a plan
    assert _attn([0, 10], [0], plan=cw.suffix_prefill_plan([0, 10], [0], 32, 8, 128, 2)) == E   # splits
    assert _attn([0, 10], [0], scale=float("nan")) == E
    assert _attn([0, 10], [0], scale=-1.0) == E
    assert _attn([0, 10], [0], nb=0) == E
    assert "prefix_len" in cw.last_error() or "num_blocks" in cw.last_error()
    assert _append([0, 10], [8]) == E
    assert _append([0, 10], [0], d=80) == U
    assert _append([0, 10], [0], bs=8) == U
    assert _append([0, 10], [0], hkv=0) == E
    assert _append([0, 1000], [16 * 90]) == E
    assert _attn([0, 0], [0]) == cw.CW_OK                 # nothing to do: no launch
    assert _append([0, 0], [16]) == cw.CW_OK


def _qkv(cu, plen, rope_len=4096, hidden=256, hq=8, hkv=2, d=128, bs=16, stride=100, nb=100, bias=True, x=True):
    cu_a, cu_p = _arr(cu)
    pl_a, pl_p = _arr(plen)
    d_ = _dummy()
    return cw.lib().cw_qkv_rope_append(d_ if x else None, d_, d_ if bias else None, d_, rope_len, hidden, d_, d_,
                                       d_, d_, stride, d_, d_, cu_p, pl_p, len(plen), hq, hkv, d, bs, nb, None)


def test_qkv_rope_append_validates_before_launch():
    E, U = cw.CW_EINVAL, cw.CW_EUNSUPPORTED
    assert _qkv([0, 10], [8]) == E                        # the batch checks of the append
    assert _qkv([0, 1000], [16 * 90]) == E
    assert _qkv([0, 10], [0], x=False) == E
    assert _qkv([0, 10], [0], hq=6, hkv=4) == E
    assert _qkv([0, 10], [0], nb=0) == E
    assert _qkv([0, 10], [0], d=96) == U
    assert _qkv([0, 10], [0], bs=32) == U
    assert _qkv([0, 10], [0], hidden=48) == U             # not a multiple of 32
    assert _qkv([0, 10], [0], hidden=0) == U
    assert _qkv([0, 10], [0], rope_len=-1) == E
    assert _qkv([0, 10, 20], [32, 48], rope_len=57) == E  # last position 48 + 9 = 57 needs 58 entries
    assert "rotary table" in cw.last_error()
    assert _qkv([0, 0], [16], rope_len=0) == cw.CW_OK      # nothing to do: no launch
    assert _qkv([0, 0, 0], [16, 32], rope_len=0, bias=False) == cw.CW_OK


def _split(cu, plen, splits=2, ws_bytes=None, hq=32, hkv=8, d=128, workspace=True):
    try:
        plan = cw.suffix_prefill_plan(cu, plen, hq, hkv, d if d in (64, 128) else 128, splits)
    except cw.CwError:
        return cw.CW_EINVAL if not (1 <= splits <= 64) else None
    return _attn(cu, plen, hq=hq, hkv=hkv, d=d, plan=plan, split=True, ws_bytes=ws_bytes, workspace=workspace)


def test_split_workspace_size():
    f = cw.lib().cw_suffix_prefill_split_workspace_bytes
    # parts of O (fp32) for every (row, head), then one fp32 log-sum-exp per (row, head)
    n = f(100, 32, 128, 3)
    o_bytes = 3 * 100 * 32 * 128 * 4
    assert n == -(-o_bytes // 256) * 256 + 3 * 100 * 32 * 4
    assert f(0, 32, 128, 1) == 0
    assert f(10, 32, 96, 1) == cw.CW_EINVAL and f(10, 32, 128, 0) == cw.CW_EINVAL
    assert f(10, 32, 128, 65) == cw.CW_EINVAL and f(-1, 32, 128, 1) == cw.CW_EINVAL


def test_split_and_merge_validate_before_launch():
    E, U = cw.CW_EINVAL, cw.CW_EUNSUPPORTED
    assert _split([0, 10], [8]) == E                       # the same batch checks as the plain call
    assert _split([0, 10], [0], d=96) == U
    assert _split([0, 10], [0], splits=0) == E
    assert _split([0, 10], [0], splits=65) == E
    assert _split([0, 10], [0], ws_bytes=16) == E          # workspace too small
    assert "workspace" in cw.last_error()
    assert _split([0, 10], [0], workspace=False) == E
    d_ = _dummy()
    merge = cw.lib().cw_lse_merge
    assert merge(d_, d_, 0, 10, 128, d_, None) == E
    assert merge(None, d_, 2, 10, 128, d_, None) == E
    assert merge(d_, d_, 2, -1, 128, d_, None) == E
    assert merge(d_, d_, 2, 10, 12, d_, None) == U
    assert merge(d_, d_, 2, 0, 128, d_, None) == cw.CW_OK   # no rows: no launch


def test_host_calls_reject_bad_arguments():
    with pytest.raises(cw.CwError):
        cw.Pool(0)
    with pytest.raises(cw.CwError):
        cw.Pool(3, [0, 0, 1])
    p = cw.Pool(4)
    with pytest.raises(cw.CwError) as e:
        p.alloc(5)
    assert e.value.status == cw.CW_ENOSPC and p.num_free == 4
    with pytest.raises(cw.CwError):
        p.release([0])
    a = p.alloc(2)
    with pytest.raises(cw.CwError):
        p.commit([5, 6], [a[0], a[0]])
    with pytest.raises(cw.CwError):
        cw.suffix_prefill_plan([0, 10], [0], 32, 8, 96)


def test_probe_mfma_flops_and_argument_errors():
    # FLOPs of one call: 8 waves x iters x 8 instructions x 2*32*32*16 per workgroup
    assert cw.probe_mfma_bf16_flops(1, 1) == 8 * 8 * 32768
    assert cw.probe_mfma_bf16_flops(2000, 1024) == 1024 * 8 * 2000 * 8 * 32768
    with pytest.raises(ValueError):
        cw.probe_mfma_bf16_flops(0, 1)
    lib = cw.lib()
    dummy = ctypes.c_void_p(16)   # never dereferenced: every case fails its checks first
    assert lib.cw_probe_mfma_bf16(None, 8192, dummy, 1, 1, None) == cw.CW_EINVAL
    assert lib.cw_probe_mfma_bf16(dummy, 8192, None, 1, 1, None) == cw.CW_EINVAL
    assert lib.cw_probe_mfma_bf16(dummy, 5120, dummy, 1, 1, None) == cw.CW_EINVAL    # < 6 fragments
    assert lib.cw_probe_mfma_bf16(dummy, 8193, dummy, 1, 1, None) == cw.CW_EINVAL    # not whole fragments
    assert lib.cw_probe_mfma_bf16(dummy, 8192, dummy, 0, 1, None) == cw.CW_EINVAL
    assert lib.cw_probe_mfma_bf16(dummy, 8192, dummy, 1, 0, None) == cw.CW_EINVAL
    assert "probe_mfma_bf16" in cw.last_error()


def test_debug_check_of_device_copies():
    # CPU tensors stand in for the device copies: the check compares values only
    bt = np.array([[3, 1, 0, -1], [2, 4, -1, -1]], dtype=np.int32)
    meta = cw.BatchMeta(bt, [0, 20, 30], [32, 16], 4, 1, 64, device=None)
    import torch
    meta.bt, meta.cu, meta.plen = (torch.from_numpy(a.copy()) for a in (meta.bt_host, meta.cu_host, meta.plen_host))
    meta.plan = torch.from_numpy(meta.plan_host.copy())
    meta.check_device_copies()
    meta.cu[2] = 31
    with pytest.raises(ValueError, match="cu_suffix"):
        meta.check_device_copies()
    meta.cu[2] = 30
    meta.plan[20] += 1
    with pytest.raises(ValueError, match="plan"):
        meta.check_device_copies()
    meta.plan = None
    with pytest.raises(ValueError, match="no device copy"):
        meta.check_device_copies()


# ------------------------------------------------------------------ fused append + attention plan
def _expected_append_table(cu, plen, bt, nb):
    """The (source, destination) words by their definition, from the batch
    description alone: a request's own suffix blocks are read from its rows and
    written to their block; a prefix block that is a full suffix block of the
    batch is read from that block's rows; other in-pool blocks from the cache."""
    B, stride = bt.shape
    fresh = {}
    for r in range(B):
        P, L = plen[r], plen[r] + cu[r + 1] - cu[r]
        for j in range(P // 16, -(-L // 16)):
            if 0 <= bt[r, j] < nb:
                fresh[int(bt[r, j])] = cu[r] + 16 * j - P if 16 * (j + 1) <= L else None
    rows = lambda R: int(np.array([0x80000000 | int(R)], np.uint32).view(np.int32)[0])   # noqa: E731
    t = np.full((B, stride, 2), -1, np.int64)
    for r in range(B):
        P, L = plen[r], plen[r] + cu[r + 1] - cu[r]
        for j in range(-(-L // 16)):
            b = int(bt[r, j])
            if not 0 <= b < nb:
                continue
            if j >= P // 16:
                t[r, j] = (rows(cu[r] + 16 * j - P), b)
            else:
                t[r, j, 0] = rows(fresh[b]) if b in fresh else 16 * b
    return t


def _random_batch(rng, B=6, stride=12, nb=200):
    S = rng.integers(0, 60, size=B)
    P = 16 * rng.integers(0, 4, size=B)
    cu = np.concatenate([[0], np.cumsum(S)]).astype(np.int32)
    bt = rng.permutation(nb)[:B * stride].reshape(B, stride).astype(np.int32)
    return cu, P.astype(np.int32), bt


def test_append_plan_table_matches_its_definition():
    rng = np.random.default_rng(3)
    for trial in range(20):
        cu, P, bt = _random_batch(rng)
        nb = 200
        # alias some prefix blocks to full suffix blocks of the batch, and put
        # out-of-pool entries in prefix and suffix blocks
        full = [(r, j) for r in range(len(P)) for j in range(P[r] // 16, (P[r] + cu[r + 1] - cu[r]) // 16)]
        pre = [(r, j) for r in range(len(P)) for j in range(P[r] // 16)]
        for (r, j), (r2, j2) in zip(pre[:2], full[::-1][:2]):
            if r != r2:
                bt[r, j] = bt[r2, j2]
        if trial % 3 == 0 and pre:
            bt[pre[-1]] = -1
        if trial % 4 == 1 and full:
            bt[full[0]] = nb + 3
        plan = cw.suffix_prefill_append_plan(cu, P, bt, 8, 2, 128, nb)
        assert plan[cw.HDR_TABLE] > 0 and plan[cw.HDR_TABLE_STRIDE] == bt.shape[1] and plan[cw.HDR_NUM_BLOCKS] == nb
        np.testing.assert_array_equal(cw.append_table(plan), _expected_append_table(cu, P, bt, nb))
        # the entries are those of the unsplit plan
        np.testing.assert_array_equal(cw.plan_entries(plan)[:, :12],
                                      cw.plan_entries(cw.suffix_prefill_plan(cu, P, 8, 2, 128))[:, :12])


def test_append_plan_refuses_racing_or_mixed_blocks():
    cu = np.array([0, 40, 70], np.int32)
    P = np.array([32, 16], np.int32)
    bt = np.arange(2 * 8, dtype=np.int32).reshape(2, 8) + 10
    bt2 = bt.copy()
    bt2[1, 2] = bt2[0, 3]                       # a suffix block named twice
    with pytest.raises(cw.CwError) as ei:
        cw.suffix_prefill_append_plan(cu, P, bt2, 8, 2, 128, 100)
    assert ei.value.status == cw.CW_EINVAL
    bt3 = bt.copy()
    bt3[1, 0] = bt3[0, 4]                       # request 0's partial last block (keys 64..71)
    with pytest.raises(cw.CwError) as ei:
        cw.suffix_prefill_append_plan(cu, P, bt3, 8, 2, 128, 100)
    assert ei.value.status == cw.CW_EUNSUPPORTED
    bt4 = bt.copy()
    bt4[1, 0] = bt4[0, 3]                       # a full suffix block: allowed, read from its rows
    t = cw.append_table(cw.suffix_prefill_append_plan(cu, P, bt4, 8, 2, 128, 100))
    assert tuple(t[1, 0]) == (int(np.array([0x80000000 | 16], np.uint32).view(np.int32)[0]), -1)
    with pytest.raises(cw.CwError):
        cw.suffix_prefill_append_plan(cu, P, bt, 8, 2, 128, 0)        # num_blocks
    with pytest.raises(cw.CwError):
        cw.suffix_prefill_append_plan(cu, P, bt[:, :4], 8, 2, 128, 100)   # stride too small for request 0


def _fused_call(cu, plen, bt, plan, hq=8, hkv=2, d=128, nb=100, bt_call=None):
    cu_a, cu_p = _arr(cu)
    pl_a, pl_p = _arr(plen)
    b = np.ascontiguousarray(bt if bt_call is None else bt_call, np.int32)
    bp = b.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    plan = np.ascontiguousarray(plan, np.int32)
    pp = plan.ctypes.data_as(ctypes.POINTER(ctypes.c_int32))
    d_ = _dummy()
    return cw.lib().cw_suffix_prefill_append_attn(d_, d_, d_, d_, d_, bp, b.shape[1], cu_p, pl_p, len(plen), hq, hkv,
                                                  d, 16, nb, 0.1, pp, d_, d_, None)


def test_fused_call_validates_its_plan_before_launch():
    E = cw.CW_EINVAL
    cu = np.array([0, 40, 70], np.int32)
    P = np.array([32, 16], np.int32)
    bt = np.arange(2 * 8, dtype=np.int32).reshape(2, 8) + 10
    fused = cw.suffix_prefill_append_plan(cu, P, bt, 8, 2, 128, 100)
    plain = cw.suffix_prefill_plan(cu, P, 8, 2, 128)
    assert _fused_call(cu, P, bt, plain) == E                          # no table
    assert "append table" in cw.last_error()
    other = bt.copy()
    other[0, 0] = 99
    assert _fused_call(cu, P, bt, fused, bt_call=other) == E           # another block table
    assert _fused_call(cu, P, bt, fused, nb=101) == E                  # another pool size
    assert _fused_call(cu, P, bt, fused, hq=16) == E                   # another head count
    assert _attn(cu, P, hq=8, hkv=2, stride=8, plan=fused) == E        # the plain call refuses it
    assert "cw_suffix_prefill_append_attn" in cw.last_error()
    assert _fused_call([0, 0], [16], bt[:1], cw.suffix_prefill_append_plan([0, 0], [16], bt[:1], 8, 2, 128, 100)) \
        == cw.CW_OK                                                    # nothing to do: no launch
