"""Places a synthetic workload in GPU memory for the library's device calls.

Set-up only: it schedules each batch through the library's block pool (chained
hashes, prefix match, allocation, commit), draws the K/V/Q values from
`inputs`, and writes the cached prefix blocks of every request into the paged
caches as the state they would be in after earlier requests were served.
Every cache element no request references holds a NaN sentinel, so a kernel
that read past a prompt's end would show it.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np
import torch

from . import cw
from .workload import Workload, logical_kv, suffix_q

SENTINEL_BITS = 0x7FC1  # a quiet-NaN bfloat16 pattern


@dataclass
class Scheduled:
    """Host description of a scheduled batch (int32 arrays)."""
    block_table: np.ndarray
    prefix_len: np.ndarray
    cu_suffix: np.ndarray
    num_blocks: int
    pool: object = None

    @property
    def suffix_len(self) -> np.ndarray:
        return np.diff(self.cu_suffix)


def bt_stride_for(w: Workload) -> int:
    return max(math.ceil(p.length / w.block_size) for p in w.prompts + w.warmup)


def schedule(w: Workload, pool: "cw.Pool | None" = None) -> Scheduled:
    """Runs the workload's host path through libcw's pool.

    Trace workloads serve their warm-up prompts one by one (schedule, then
    release), then schedule the batch in one call, so each request's cached
    depth is whatever the pool matches. Workloads with fixed depths allocate
    each prompt's blocks in the pool's placement order and take the given
    depths.
    """
    nb = w.num_blocks()
    if pool is None:
        pool = cw.Pool(nb, w.free_order())
    stride = bt_stride_for(w)
    if w.prefix_lens is None:
        for p in w.warmup:
            bt, pl, cu = cw.schedule_batch(pool, [p.tokens(w.seed)], stride, w.block_size)
            cw.release_batch(pool, bt, pl, cu, w.block_size)
        bt, pl, cu = cw.schedule_batch(pool, [p.tokens(w.seed) for p in w.prompts], stride, w.block_size)
        return Scheduled(bt, pl, cu, nb, pool)
    bt = np.full((w.batch, stride), -1, dtype=np.int32)
    for r, p in enumerate(w.prompts):
        n = math.ceil(p.length / w.block_size)
        bt[r, :n] = pool.alloc(n)
    pl = np.asarray(w.prefix_lens, dtype=np.int32)
    S = np.array([p.length for p in w.prompts]) - pl
    cu = np.concatenate([[0], np.cumsum(S)]).astype(np.int32)
    return Scheduled(bt, pl, cu, nb, pool)


@dataclass
class DeviceBatch:
    workload: Workload
    sched: Scheduled
    meta: "cw.BatchMeta"
    q: torch.Tensor
    k_new: torch.Tensor
    v_new: torch.Tensor
    k_cache: torch.Tensor
    v_cache: torch.Tensor
    logical_k: list | None = None   # per request [L, Hkv, D] bf16 (host), when kept
    logical_v: list | None = None
    q_host: list | None = None      # per request [S, Hq, D] bf16 (host), when kept

    @property
    def scale(self) -> float:
        return self.workload.scale


def _blocks_view(x: torch.Tensor, block_size: int) -> torch.Tensor:
    """[n * bs, Hkv, D] -> [n, Hkv, bs, D]"""
    n = x.shape[0] // block_size
    return x[:n * block_size].reshape(n, block_size, x.shape[1], x.shape[2]).permute(0, 2, 1, 3)


def materialize(w: Workload, device="cuda", keep_host=None, gen_device=None,
                sched: Scheduled | None = None) -> DeviceBatch:
    """Schedules `w` (unless `sched` is given) and fills the device buffers.

    keep_host: request indices whose logical K/V and suffix Q are also kept on
    the host (None = all). gen_device: where values are drawn ("cpu" by
    default; "cuda" for large batches)."""
    if sched is None:
        sched = schedule(w)
    gen = gen_device or "cpu"
    bs, hkv, hq, D = w.block_size, w.num_kv_heads, w.num_q_heads, w.head_dim
    keep = set(range(w.batch)) if keep_host is None else set(keep_host)
    k_cache = torch.full((sched.num_blocks, hkv, bs, D), 0, dtype=torch.int16, device=device)
    k_cache.fill_(SENTINEL_BITS)
    k_cache = k_cache.view(torch.bfloat16)
    v_cache = k_cache.clone()
    total = int(sched.cu_suffix[-1])
    q = torch.empty((total, hq, D), dtype=torch.bfloat16, device=device)
    k_new = torch.empty((total, hkv, D), dtype=torch.bfloat16, device=device)
    v_new = torch.empty((total, hkv, D), dtype=torch.bfloat16, device=device)
    lk, lv, qh = {}, {}, {}
    for r, prompt in enumerate(w.prompts):
        P = int(sched.prefix_len[r])
        c0, c1 = int(sched.cu_suffix[r]), int(sched.cu_suffix[r + 1])
        k, v = logical_kv(w, prompt, gen)
        qs = suffix_q(w, prompt, P, gen)
        q[c0:c1] = qs.to(device)
        k_new[c0:c1] = k[P:].to(device)
        v_new[c0:c1] = v[P:].to(device)
        nblk = P // bs
        if nblk:
            ids = torch.from_numpy(sched.block_table[r, :nblk].astype(np.int64)).to(device)
            k_cache[ids] = _blocks_view(k[:P], bs).to(device)
            v_cache[ids] = _blocks_view(v[:P], bs).to(device)
        if r in keep:
            lk[r], lv[r], qh[r] = k.cpu(), v.cpu(), qs.cpu()
    meta = cw.BatchMeta(sched.block_table, sched.cu_suffix, sched.prefix_len, hq, hkv, D, device)
    return DeviceBatch(w, sched, meta, q, k_new, v_new, k_cache, v_cache,
                       [lk.get(r) for r in range(w.batch)], [lv.get(r) for r in range(w.batch)],
                       [qh.get(r) for r in range(w.batch)])
