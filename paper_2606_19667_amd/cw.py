"""Python binding of libcw (include/cw.h): argument marshalling only.

Every function here checks and converts its arguments, then calls the C entry
point of the same name; all computation happens in the library (host C++ for
hashing, the block pool and planning; HIP kernels on the GPU for the append and
the attention). torch tensors provide device memory and the HIP stream.

The library is loaded after torch so that both use the one HIP runtime that
torch has already loaded. A missing library raises at import time: there is no
fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

# CW_LIBRARY may name another build of the same library (the sanitizer build)
LIB_PATH = os.environ.get("CW_LIBRARY") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libcw.so")

CW_OK = 0
CW_EINVAL = -1
CW_EUNSUPPORTED = -2
CW_ENOSPC = -3
CW_EHIP = -4
BLOCK_SIZE = 16
TILE_ROWS = 256    # packed query rows (heads x positions) of one attention tile (cw.h)
PLAN_HEADER = 16   # int32 words of a plan's header, then entries of PLAN_ENTRY words
PLAN_ENTRY = 16
HDR_ENTRIES, HDR_GRID, HDR_SPLITS, HDR_QUEUE_LEN, HDR_WORK = 1, 4, 5, 11, 12
HDR_TABLE, HDR_TABLE_STRIDE, HDR_NUM_BLOCKS = 13, 14, 15
ENT_R, ENT_G, ENT_ROW0, ENT_NVALID, ENT_CU0, ENT_P, ENT_L, ENT_KBEG, ENT_KEND, ENT_SPLIT = range(10)

_i32 = ctypes.c_int32
_i64 = ctypes.c_int64
_f32 = ctypes.c_float
_vp = ctypes.c_void_p
_pi32 = ctypes.POINTER(ctypes.c_int32)
_pi64 = ctypes.POINTER(ctypes.c_int64)
_pu64 = ctypes.POINTER(ctypes.c_uint64)


class CwError(RuntimeError):
    """A libcw call returned a non-OK status."""

    def __init__(self, status: int, message: str):
        super().__init__(f"libcw status {status}: {message}")
        self.status = status


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_19667_amd.build`")
    lib = ctypes.CDLL(LIB_PATH)
    sig = {
        "cw_abi_version": (_i32, []),
        "cw_last_error": (ctypes.c_char_p, []),
        "cw_block_hashes": (_i32, [_pi32, _i64, _i32, _pu64]),
        "cw_pool_create": (_i32, [_i32, _pi32, ctypes.POINTER(_vp)]),
        "cw_pool_destroy": (None, [_vp]),
        "cw_pool_clone": (_i32, [_vp, ctypes.POINTER(_vp)]),
        "cw_pool_num_free": (_i32, [_vp]),
        "cw_prefix_match": (_i32, [_vp, _pu64, _i32, _i32, _pi32, _pi32]),
        "cw_pool_alloc": (_i32, [_vp, _i32, _pi32]),
        "cw_pool_commit": (_i32, [_vp, _pu64, _pi32, _i32]),
        "cw_pool_release": (_i32, [_vp, _pi32, _i32]),
        "cw_schedule_batch": (_i32, [_vp, _pi32, _pi64, _i32, _i32, _i32, _pi32, _pi32, _pi32]),
        "cw_release_batch": (_i32, [_vp, _pi32, _i32, _pi32, _pi32, _i32, _i32]),
        "cw_kv_append": (_i32, [_vp, _vp, _vp, _vp, _vp, _i32, _vp, _vp, _pi32, _pi32,
                                _i32, _i32, _i32, _i32, _i32, _vp]),
        "cw_suffix_prefill_plan_words": (_i64, [_pi32, _pi32, _i32, _i32, _i32, _i32, _i32]),
        "cw_suffix_prefill_plan": (_i32, [_pi32, _pi32, _i32, _i32, _i32, _i32, _i32, _pi32, _i64]),
        "cw_suffix_prefill_attn": (_i32, [_vp, _vp, _vp, _vp, _i32, _vp, _vp, _pi32, _pi32,
                                          _i32, _i32, _i32, _i32, _i32, _i32, _f32, _pi32, _vp,
                                          _vp, _vp]),
        "cw_suffix_prefill_append_plan_words": (_i64, [_pi32, _pi32, _i32, _i32, _i32, _i32, _i32]),
        "cw_suffix_prefill_append_plan": (_i32, [_pi32, _pi32, _pi32, _i32, _i32, _i32, _i32, _i32, _i32,
                                                 _pi32, _i64]),
        "cw_suffix_prefill_append_attn": (_i32, [_vp, _vp, _vp, _vp, _vp, _pi32, _i32, _pi32, _pi32, _i32,
                                                 _i32, _i32, _i32, _i32, _i32, _f32, _pi32, _vp, _vp, _vp]),
        "cw_suffix_prefill_split_workspace_bytes": (_i64, [_i64, _i32, _i32, _i32]),
        "cw_suffix_prefill_attn_split": (_i32, [_vp, _vp, _vp, _vp, _i32, _vp, _vp, _pi32, _pi32,
                                                _i32, _i32, _i32, _i32, _i32, _i32, _f32, _pi32, _vp,
                                                _vp, _i64, _vp, _vp]),
        "cw_lse_merge": (_i32, [_vp, _vp, _i32, _i64, _i32, _vp, _vp]),
        "cw_noalloc_scratch_bytes": (_i64, []),
        "cw_suffix_prefill_attn_split_noalloc": (_i32, [_vp, _vp, _vp, _vp, _i32, _vp, _vp, _pi32, _pi32,
                                                        _i32, _i32, _i32, _i32, _i32, _i32, _f32, _pi32, _vp,
                                                        _vp, _vp]),
        "cw_tree_create": (_i32, [_i32, ctypes.POINTER(_vp)]),
        "cw_tree_destroy": (None, [_vp]),
        "cw_tree_num_nodes": (_i64, [_vp]),
        "cw_tree_insert": (_i32, [_vp, _pi64, _i32]),
        "cw_tree_mark_stale": (_i32, [_vp, _pi64, _i32, _i32]),
        "cw_tree_order": (_i32, [_vp, _i32, _pi64, _i32, _pi64, _pi32, _pi32]),
        "cw_rope_table": (_i32, [_i32, _i32, ctypes.c_double, ctypes.POINTER(ctypes.c_float)]),
        "cw_qkv_rope_append": (_i32, [_vp, _vp, _vp, _vp, _i32, _i32, _vp, _vp, _vp, _vp, _i32, _vp, _vp,
                                      _pi32, _pi32, _i32, _i32, _i32, _i32, _i32, _i32, _vp]),
        "cw_probe_mfma_bf16_flops": (_i64, [_i32, _i32]),
        "cw_probe_mfma_bf16": (_i32, [_vp, _i64, _vp, _i32, _i32, _vp]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


_lib = _load()

EXPORTED = ("cw_abi_version", "cw_last_error", "cw_block_hashes", "cw_pool_create",
            "cw_pool_destroy", "cw_pool_clone", "cw_pool_num_free", "cw_prefix_match",
            "cw_pool_alloc", "cw_pool_commit", "cw_pool_release", "cw_schedule_batch",
            "cw_release_batch", "cw_kv_append", "cw_suffix_prefill_plan_words",
            "cw_suffix_prefill_plan", "cw_suffix_prefill_attn", "cw_suffix_prefill_append_plan_words",
            "cw_suffix_prefill_append_plan", "cw_suffix_prefill_append_attn",
            "cw_suffix_prefill_split_workspace_bytes", "cw_suffix_prefill_attn_split", "cw_lse_merge",
            "cw_noalloc_scratch_bytes", "cw_suffix_prefill_attn_split_noalloc",
            "cw_tree_create", "cw_tree_destroy", "cw_tree_num_nodes", "cw_tree_insert",
            "cw_tree_mark_stale", "cw_tree_order", "cw_rope_table", "cw_qkv_rope_append",
            "cw_probe_mfma_bf16_flops", "cw_probe_mfma_bf16")


def lib() -> ctypes.CDLL:
    return _lib


def abi_version() -> int:
    return int(_lib.cw_abi_version())


def last_error() -> str:
    return _lib.cw_last_error().decode()


def _check(status: int) -> None:
    if status != CW_OK:
        raise CwError(int(status), last_error())


def _i32_array(x, name: str) -> np.ndarray:
    a = np.ascontiguousarray(np.asarray(x), dtype=np.int32)
    return a


def _ptr(a: np.ndarray, ctype):
    return a.ctypes.data_as(ctypes.POINTER(ctype)) if a.size else None


# ---------------------------------------------------------------- host calls
def block_hashes(tokens, block_size: int = BLOCK_SIZE) -> np.ndarray:
    """cw_block_hashes: chained hashes of the full blocks (uint64 array)."""
    t = _i32_array(tokens, "tokens")
    out = np.zeros(len(t) // block_size, dtype=np.uint64)
    _check(_lib.cw_block_hashes(_ptr(t, ctypes.c_int32), len(t), block_size, _ptr(out, ctypes.c_uint64)))
    return out


class Pool:
    """Owner of a cw_pool handle (host-side block bookkeeping)."""

    def __init__(self, num_blocks: int | None = None, free_order=None, _handle=None):
        if _handle is not None:
            self._h = _handle
            return
        h = _vp()
        fo = None if free_order is None else _i32_array(free_order, "free_order")
        if fo is not None and len(fo) != num_blocks:
            raise ValueError("free_order must have num_blocks entries")
        _check(_lib.cw_pool_create(int(num_blocks), None if fo is None else _ptr(fo, ctypes.c_int32),
                                   ctypes.byref(h)))
        self._h = h

    @property
    def handle(self):
        return self._h

    def close(self) -> None:
        if self._h is not None and self._h.value:
            _lib.cw_pool_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def clone(self) -> "Pool":
        h = _vp()
        _check(_lib.cw_pool_clone(self._h, ctypes.byref(h)))
        return Pool(_handle=h)

    @property
    def num_free(self) -> int:
        return int(_lib.cw_pool_num_free(self._h))

    def prefix_match(self, hashes, max_match: int) -> np.ndarray:
        hs = np.ascontiguousarray(hashes, dtype=np.uint64)
        ids = np.zeros(len(hs), dtype=np.int32)
        depth = ctypes.c_int32(0)
        _check(_lib.cw_prefix_match(self._h, _ptr(hs, ctypes.c_uint64), len(hs), int(max_match),
                                    _ptr(ids, ctypes.c_int32), ctypes.byref(depth)))
        return ids[:depth.value].copy()

    def alloc(self, n: int) -> np.ndarray:
        ids = np.zeros(max(0, int(n)), dtype=np.int32)
        _check(_lib.cw_pool_alloc(self._h, int(n), _ptr(ids, ctypes.c_int32)))
        return ids

    def commit(self, hashes, block_ids) -> None:
        hs = np.ascontiguousarray(hashes, dtype=np.uint64)
        ids = _i32_array(block_ids, "block_ids")
        if len(hs) != len(ids):
            raise ValueError("hashes and block_ids differ in length")
        _check(_lib.cw_pool_commit(self._h, _ptr(hs, ctypes.c_uint64), _ptr(ids, ctypes.c_int32), len(ids)))

    def release(self, block_ids) -> None:
        ids = _i32_array(block_ids, "block_ids")
        _check(_lib.cw_pool_release(self._h, _ptr(ids, ctypes.c_int32), len(ids)))


ORDER_RETRIEVAL, ORDER_SORTED, ORDER_RECENCY, ORDER_GREEDY, ORDER_EXHAUSTIVE = 0, 1, 2, 3, 4
ORDER_NAMES = {"retrieval": ORDER_RETRIEVAL, "sorted": ORDER_SORTED, "recency": ORDER_RECENCY,
               "greedy": ORDER_GREEDY, "exhaustive": ORDER_EXHAUSTIVE}


def _docs_array(docs) -> np.ndarray:
    return np.ascontiguousarray(np.asarray(list(docs), dtype=np.int64).reshape(-1))


class KnowledgeTree:
    """Owner of a cw_tree handle: the trie of recently served document orders
    with the greedy walk, the exhaustive argmax and the baseline orders."""

    def __init__(self, window: int = 32):
        h = _vp()
        _check(_lib.cw_tree_create(int(window), ctypes.byref(h)))
        self._h = h
        self.window = int(window)

    def close(self) -> None:
        if self._h is not None and self._h.value:
            _lib.cw_tree_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def insert(self, order) -> None:
        """Record a served order."""
        a = _docs_array(order)
        _check(_lib.cw_tree_insert(self._h, _ptr(a, ctypes.c_int64), len(a)))

    def mark_stale(self, order, observed_depth: int) -> None:
        """Mark the nodes of `order` deeper than `observed_depth` stale."""
        a = _docs_array(order)
        _check(_lib.cw_tree_mark_stale(self._h, _ptr(a, ctypes.c_int64), len(a), int(observed_depth)))

    def order(self, docs, strategy=ORDER_GREEDY):
        """Returns (order, depth, probes) for the retrieved set `docs` (in
        retrieval rank); strategy is a CW_ORDER_* value or its name."""
        if isinstance(strategy, str):
            strategy = ORDER_NAMES[strategy]
        a = _docs_array(docs)
        out = np.zeros(len(a), dtype=np.int64)
        depth, probes = ctypes.c_int32(0), ctypes.c_int32(0)
        _check(_lib.cw_tree_order(self._h, int(strategy), _ptr(a, ctypes.c_int64), len(a),
                                  _ptr(out, ctypes.c_int64), ctypes.byref(depth), ctypes.byref(probes)))
        return [int(x) for x in out], depth.value, probes.value

    def num_nodes(self) -> int:
        return int(_lib.cw_tree_num_nodes(self._h))


def rope_table(n_positions: int, head_dim: int, base: float) -> np.ndarray:
    """cos/sin of p * theta_j for p < n_positions, j < head_dim / 2: fp32 [n, D/2, 2]."""
    out = np.empty((max(int(n_positions), 0), int(head_dim) // 2, 2), dtype=np.float32)
    _check(_lib.cw_rope_table(int(n_positions), int(head_dim), float(base),
                              out.ctypes.data_as(ctypes.POINTER(ctypes.c_float))))
    return out


def schedule_batch(pool: Pool, prompts, bt_stride: int, block_size: int = BLOCK_SIZE):
    """cw_schedule_batch over a list of token arrays.

    Returns (block_table [B, bt_stride], prefix_len [B], cu_suffix [B + 1]) as int32."""
    toks = [_i32_array(p, "tokens") for p in prompts]
    cu_tokens = np.zeros(len(toks) + 1, dtype=np.int64)
    cu_tokens[1:] = np.cumsum([len(t) for t in toks])
    flat = np.ascontiguousarray(np.concatenate(toks) if toks else np.zeros(0, np.int32), dtype=np.int32)
    B = len(toks)
    bt = np.zeros((B, bt_stride), dtype=np.int32)
    plen = np.zeros(B, dtype=np.int32)
    cu = np.zeros(B + 1, dtype=np.int32)
    _check(_lib.cw_schedule_batch(pool.handle, _ptr(flat, ctypes.c_int32), _ptr(cu_tokens, ctypes.c_int64),
                                  B, block_size, bt_stride, _ptr(bt, ctypes.c_int32),
                                  _ptr(plen, ctypes.c_int32), _ptr(cu, ctypes.c_int32)))
    return bt, plen, cu


def release_batch(pool: Pool, block_table, prefix_len, cu_suffix, block_size: int = BLOCK_SIZE) -> None:
    bt = _i32_array(block_table, "block_table")
    plen = _i32_array(prefix_len, "prefix_len")
    cu = _i32_array(cu_suffix, "cu_suffix")
    _check(_lib.cw_release_batch(pool.handle, _ptr(bt, ctypes.c_int32), bt.shape[1], _ptr(plen, ctypes.c_int32),
                                 _ptr(cu, ctypes.c_int32), len(plen), block_size))


def suffix_prefill_plan(cu_suffix, prefix_len, num_q_heads: int, num_kv_heads: int, head_dim: int,
                        num_splits: int = 1) -> np.ndarray:
    """cw_suffix_prefill_plan: the plan (int32 array: header, then entries)."""
    cu = _i32_array(cu_suffix, "cu_suffix")
    plen = _i32_array(prefix_len, "prefix_len")
    B = len(plen)
    words = int(_lib.cw_suffix_prefill_plan_words(_ptr(cu, ctypes.c_int32), _ptr(plen, ctypes.c_int32), B,
                                                  num_q_heads, num_kv_heads, head_dim, int(num_splits)))
    if words < 0:
        _check(words)
    plan = np.zeros(words, dtype=np.int32)
    _check(_lib.cw_suffix_prefill_plan(_ptr(cu, ctypes.c_int32), _ptr(plen, ctypes.c_int32), B, num_q_heads,
                                       num_kv_heads, head_dim, int(num_splits), _ptr(plan, ctypes.c_int32),
                                       len(plan)))
    return plan


def plan_entries(plan: np.ndarray) -> np.ndarray:
    """The entries of a plan as an [n, PLAN_ENTRY] view (padding included:
    entries with request -1 end a queue)."""
    n = int(plan[HDR_ENTRIES])
    return plan[PLAN_HEADER:PLAN_HEADER + n * PLAN_ENTRY].reshape(-1, PLAN_ENTRY)


def suffix_prefill_append_plan(cu_suffix, prefix_len, block_table, num_q_heads: int, num_kv_heads: int,
                               head_dim: int, num_blocks: int) -> np.ndarray:
    """cw_suffix_prefill_append_plan: the plan of the fused append + attention
    call (header, entries, then the (source, destination) table)."""
    cu = _i32_array(cu_suffix, "cu_suffix")
    plen = _i32_array(prefix_len, "prefix_len")
    bt = _i32_array(block_table, "block_table")
    if bt.ndim != 2 or bt.shape[0] != len(plen):
        raise ValueError("block_table must be [batch, stride]")
    B = len(plen)
    words = int(_lib.cw_suffix_prefill_append_plan_words(_ptr(cu, ctypes.c_int32), _ptr(plen, ctypes.c_int32),
                                                         bt.shape[1], B, num_q_heads, num_kv_heads, head_dim))
    if words < 0:
        _check(words)
    plan = np.zeros(words, dtype=np.int32)
    _check(_lib.cw_suffix_prefill_append_plan(_ptr(cu, ctypes.c_int32), _ptr(plen, ctypes.c_int32),
                                              _ptr(bt, ctypes.c_int32), bt.shape[1], B, num_q_heads, num_kv_heads,
                                              head_dim, int(num_blocks), _ptr(plan, ctypes.c_int32), len(plan)))
    return plan


def append_table(plan: np.ndarray) -> np.ndarray:
    """The (source, destination) table of a fused plan as [batch, stride, 2]."""
    t0, stride = int(plan[HDR_TABLE]), int(plan[HDR_TABLE_STRIDE])
    if t0 == 0:
        raise ValueError("not a plan of cw_suffix_prefill_append_plan")
    return plan[t0:].reshape(-1, stride, 2)


# ---------------------------------------------------------------- device calls
def _dev(t: torch.Tensor, dtype, name: str) -> int:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch tensor")
    if t.device.type != "cuda":
        raise ValueError(f"{name} must be in GPU memory")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t.data_ptr()


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return int(stream.cuda_stream)


# Debug mode: every device call first checks that the device copies of the
# batch description (block table, offsets, prefix lengths, plan) equal the host
# copies that validated it. The check synchronises the device; off by default.
# (Without it the library still refuses a host plan built for another batch,
# and the kernels compute nothing for a device plan whose header differs.)
DEBUG_CHECK_COPIES = os.environ.get("CW_DEBUG_CHECK_COPIES", "") not in ("", "0")


def _check_copies(pairs) -> None:
    """Raises ValueError naming the first (name, device tensor, host array)
    whose device copy is missing or differs from the host copy."""
    if torch.cuda.is_available():
        torch.cuda.synchronize()
    for name, dev, host in pairs:
        if dev is None:
            raise ValueError(f"{name}: no device copy")
        got = dev.detach().to("cpu").numpy()
        if got.shape != host.shape or not np.array_equal(got, host):
            raise ValueError(f"{name}: the device copy differs from the host copy")


class BatchMeta:
    """Host and device copies of a ragged batch's description.

    block_table [B, stride], cu_suffix [B + 1], prefix_len [B] (int32); the
    attention plan is built on the host by the library (plans for split counts
    other than 1 are built on first use and kept). With device=None nothing is
    uploaded and the caller assigns the device tensors bt, cu, plen, plan."""

    def __init__(self, block_table, cu_suffix, prefix_len, num_q_heads: int, num_kv_heads: int,
                 head_dim: int, device="cuda"):
        self.bt_host = _i32_array(block_table, "block_table")
        self.cu_host = _i32_array(cu_suffix, "cu_suffix")
        self.plen_host = _i32_array(prefix_len, "prefix_len")
        if self.bt_host.ndim != 2 or self.bt_host.shape[0] != len(self.plen_host):
            raise ValueError("block_table must be [batch, stride]")
        if len(self.cu_host) != len(self.plen_host) + 1:
            raise ValueError("cu_suffix must have batch + 1 entries")
        self.batch = len(self.plen_host)
        self.num_q_heads, self.num_kv_heads, self.head_dim = num_q_heads, num_kv_heads, head_dim
        self.plan_host = suffix_prefill_plan(self.cu_host, self.plen_host, num_q_heads, num_kv_heads, head_dim)
        self.device = device
        self.bt = self.cu = self.plen = self.plan = None
        self._split_plans = {}
        self._append_plans = {}
        if device is not None:
            self.bt = torch.from_numpy(self.bt_host).to(device)
            self.cu = torch.from_numpy(self.cu_host).to(device)
            self.plen = torch.from_numpy(self.plen_host).to(device)
            self.plan = torch.from_numpy(self.plan_host).to(device)

    @property
    def total_rows(self) -> int:
        return int(self.cu_host[-1])

    @property
    def bt_stride(self) -> int:
        return int(self.bt_host.shape[1])

    @property
    def num_tiles(self) -> int:
        """Tiles of the batch (plan entries of the unsplit plan, padding excluded)."""
        return int((plan_entries(self.plan_host)[:, ENT_R] >= 0).sum())

    def split_plan(self, num_splits: int):
        """(host plan, device plan) for `num_splits` key runs per tile."""
        if num_splits == 1:
            return self.plan_host, self.plan
        if num_splits not in self._split_plans:
            ph = suffix_prefill_plan(self.cu_host, self.plen_host, self.num_q_heads, self.num_kv_heads,
                                     self.head_dim, num_splits)
            pd = torch.from_numpy(ph).to(self.device) if self.device is not None else None
            self._split_plans[num_splits] = (ph, pd)
        return self._split_plans[num_splits]

    def append_plan(self, num_blocks: int):
        """(host plan, device plan) of the fused append + attention call for a
        pool of `num_blocks` blocks."""
        if num_blocks not in self._append_plans:
            ph = suffix_prefill_append_plan(self.cu_host, self.plen_host, self.bt_host, self.num_q_heads,
                                            self.num_kv_heads, self.head_dim, num_blocks)
            pd = torch.from_numpy(ph).to(self.device) if self.device is not None else None
            self._append_plans[num_blocks] = (ph, pd)
        return self._append_plans[num_blocks]

    def _hp(self, a):
        return _ptr(a, ctypes.c_int32)

    def check_device_copies(self) -> None:
        """The caller guarantees that the device copies equal the host ones
        (the library validates and plans with the host copies, the kernels
        read the device copies); this checks it, synchronising the device."""
        pairs = [("block_table", self.bt, self.bt_host), ("cu_suffix", self.cu, self.cu_host),
                 ("prefix_len", self.plen, self.plen_host), ("plan", self.plan, self.plan_host)]
        for n, (ph, pd) in self._split_plans.items():
            pairs.append((f"plan ({n} splits)", pd, ph))
        for n, (ph, pd) in self._append_plans.items():
            pairs.append((f"append plan ({n} blocks)", pd, ph))
        _check_copies(pairs)


def _cache_shapes_ok(k_cache: torch.Tensor, v_cache: torch.Tensor, hkv: int, D: int) -> bool:
    """Both caches are [num_blocks, Hkv, 16, D] (block rows are tokens)."""
    return (k_cache.dim() == 4 and v_cache.dim() == 4 and tuple(k_cache.shape[1:]) == (hkv, BLOCK_SIZE, D)
            and tuple(v_cache.shape) == tuple(k_cache.shape))


def kv_append(meta: BatchMeta, k_new: torch.Tensor, v_new: torch.Tensor, k_cache: torch.Tensor,
              v_cache: torch.Tensor, stream=None) -> None:
    """cw_kv_append: write the suffix K/V rows into their cache blocks."""
    if DEBUG_CHECK_COPIES:
        meta.check_device_copies()
    hkv, D = meta.num_kv_heads, meta.head_dim
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        if tuple(t.shape) != (meta.total_rows, hkv, D):
            raise ValueError(f"{name} must be [{meta.total_rows}, {hkv}, {D}], got {tuple(t.shape)}")
    if not _cache_shapes_ok(k_cache, v_cache, hkv, D):
        raise ValueError("k_cache and v_cache must both be [num_blocks, Hkv, 16, D]")
    _check(_lib.cw_kv_append(_dev(k_new, torch.bfloat16, "k_new"), _dev(v_new, torch.bfloat16, "v_new"),
                             _dev(k_cache, torch.bfloat16, "k_cache"), _dev(v_cache, torch.bfloat16, "v_cache"),
                             _dev(meta.bt, torch.int32, "block_table"), meta.bt_stride,
                             _dev(meta.cu, torch.int32, "cu_suffix"), _dev(meta.plen, torch.int32, "prefix_len"),
                             meta._hp(meta.cu_host), meta._hp(meta.plen_host), meta.batch, hkv, D, BLOCK_SIZE,
                             k_cache.shape[0], _stream(stream)))


def qkv_rope_append(meta: BatchMeta, x: torch.Tensor, w: torch.Tensor, rope: torch.Tensor,
                    k_cache: torch.Tensor, v_cache: torch.Tensor, bias: torch.Tensor | None = None,
                    q_out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """cw_qkv_rope_append: project the suffix rows x [total_s, hidden] with w
    [(Hq + 2 Hkv) D, hidden] (+ bias), rotate q and k at their positions with
    the table rope [n, D/2, 2] (cw.rope_table on the device), write k and v into
    the cache blocks and return q_out [total_s, Hq, D] bf16."""
    if DEBUG_CHECK_COPIES:
        meta.check_device_copies()
    hq, hkv, D = meta.num_q_heads, meta.num_kv_heads, meta.head_dim
    if x.dim() != 2 or x.shape[0] != meta.total_rows:
        raise ValueError(f"x must be [{meta.total_rows}, hidden], got {tuple(x.shape)}")
    hidden = int(x.shape[1])
    nf = (hq + 2 * hkv) * D
    if tuple(w.shape) != (nf, hidden):
        raise ValueError(f"w must be [{nf}, {hidden}], got {tuple(w.shape)}")
    if bias is not None and tuple(bias.shape) != (nf,):
        raise ValueError(f"bias must be [{nf}], got {tuple(bias.shape)}")
    if rope.dim() != 3 or tuple(rope.shape[1:]) != (D // 2, 2):
        raise ValueError(f"rope must be [n, {D // 2}, 2], got {tuple(rope.shape)}")
    if not _cache_shapes_ok(k_cache, v_cache, hkv, D):
        raise ValueError("k_cache and v_cache must both be [num_blocks, Hkv, 16, D]")
    if q_out is None:
        q_out = torch.empty((meta.total_rows, hq, D), dtype=torch.bfloat16, device=x.device)
    elif tuple(q_out.shape) != (meta.total_rows, hq, D):
        raise ValueError(f"q_out must be [{meta.total_rows}, {hq}, {D}]")
    _check(_lib.cw_qkv_rope_append(
        _dev(x, torch.bfloat16, "x"), _dev(w, torch.bfloat16, "w"),
        None if bias is None else _dev(bias, torch.bfloat16, "bias"), _dev(rope, torch.float32, "rope"),
        int(rope.shape[0]), hidden, _dev(q_out, torch.bfloat16, "q_out"),
        _dev(k_cache, torch.bfloat16, "k_cache"), _dev(v_cache, torch.bfloat16, "v_cache"),
        _dev(meta.bt, torch.int32, "block_table"), meta.bt_stride,
        _dev(meta.cu, torch.int32, "cu_suffix"), _dev(meta.plen, torch.int32, "prefix_len"),
        meta._hp(meta.cu_host), meta._hp(meta.plen_host), meta.batch, hq, hkv, D, BLOCK_SIZE,
        k_cache.shape[0], _stream(stream)))
    return q_out


def suffix_prefill_attn(meta: BatchMeta, q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                        softmax_scale: float, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """cw_suffix_prefill_attn: attention of the suffix rows; returns out [total_s, Hq, D] bf16."""
    if DEBUG_CHECK_COPIES:
        meta.check_device_copies()
    hq, hkv, D = meta.num_q_heads, meta.num_kv_heads, meta.head_dim
    if tuple(q.shape) != (meta.total_rows, hq, D):
        raise ValueError(f"q must be [{meta.total_rows}, {hq}, {D}], got {tuple(q.shape)}")
    if not _cache_shapes_ok(k_cache, v_cache, hkv, D):
        raise ValueError("k_cache and v_cache must both be [num_blocks, Hkv, 16, D]")
    if out is None:
        out = torch.empty_like(q)
    elif tuple(out.shape) != tuple(q.shape):
        raise ValueError("out must have q's shape")
    _check(_lib.cw_suffix_prefill_attn(
        _dev(q, torch.bfloat16, "q"), _dev(k_cache, torch.bfloat16, "k_cache"),
        _dev(v_cache, torch.bfloat16, "v_cache"), _dev(meta.bt, torch.int32, "block_table"), meta.bt_stride,
        _dev(meta.cu, torch.int32, "cu_suffix"), _dev(meta.plen, torch.int32, "prefix_len"),
        meta._hp(meta.cu_host), meta._hp(meta.plen_host), meta.batch, hq, hkv, D, BLOCK_SIZE,
        k_cache.shape[0], float(softmax_scale), meta._hp(meta.plan_host), _dev(meta.plan, torch.int32, "plan"),
        _dev(out, torch.bfloat16, "out"), _stream(stream)))
    return out


def suffix_prefill_append_attn(meta: BatchMeta, q: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
                               k_cache: torch.Tensor, v_cache: torch.Tensor, softmax_scale: float,
                               out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """cw_suffix_prefill_append_attn: cw_kv_append and cw_suffix_prefill_attn in
    one launch (same cache image and output); returns out [total_s, Hq, D]."""
    hq, hkv, D = meta.num_q_heads, meta.num_kv_heads, meta.head_dim
    if tuple(q.shape) != (meta.total_rows, hq, D):
        raise ValueError(f"q must be [{meta.total_rows}, {hq}, {D}], got {tuple(q.shape)}")
    for name, t in (("k_new", k_new), ("v_new", v_new)):
        if tuple(t.shape) != (meta.total_rows, hkv, D):
            raise ValueError(f"{name} must be [{meta.total_rows}, {hkv}, {D}], got {tuple(t.shape)}")
    if not _cache_shapes_ok(k_cache, v_cache, hkv, D):
        raise ValueError("k_cache and v_cache must both be [num_blocks, Hkv, 16, D]")
    if out is None:
        out = torch.empty_like(q)
    elif tuple(out.shape) != tuple(q.shape):
        raise ValueError("out must have q's shape")
    ph, pd = meta.append_plan(int(k_cache.shape[0]))
    if DEBUG_CHECK_COPIES:
        meta.check_device_copies()
    _check(_lib.cw_suffix_prefill_append_attn(
        _dev(q, torch.bfloat16, "q"), _dev(k_new, torch.bfloat16, "k_new"), _dev(v_new, torch.bfloat16, "v_new"),
        _dev(k_cache, torch.bfloat16, "k_cache"), _dev(v_cache, torch.bfloat16, "v_cache"),
        meta._hp(meta.bt_host), meta.bt_stride, meta._hp(meta.cu_host), meta._hp(meta.plen_host), meta.batch,
        hq, hkv, D, BLOCK_SIZE, k_cache.shape[0], float(softmax_scale), meta._hp(ph),
        _dev(pd, torch.int32, "plan"), _dev(out, torch.bfloat16, "out"), _stream(stream)))
    return out


def split_count(meta: BatchMeta, num_cus: int = 256) -> int:
    """A split count for cw_suffix_prefill_attn_split: the most runs per tile
    for which the batch's runs still fit one per CU (one attention workgroup
    per CU): more would queue a second run on some CUs and lengthen the call
    (1 when the tiles alone fill the CUs)."""
    return max(1, min(64, num_cus // max(1, meta.num_tiles)))


def split_workspace_bytes(meta: BatchMeta, num_splits: int) -> int:
    n = _lib.cw_suffix_prefill_split_workspace_bytes(meta.total_rows, meta.num_q_heads, meta.head_dim, num_splits)
    if n < 0:
        _check(int(n))
    return int(n)


def suffix_prefill_attn_split(meta: BatchMeta, q: torch.Tensor, k_cache: torch.Tensor, v_cache: torch.Tensor,
                              softmax_scale: float, num_splits: int | None = None,
                              workspace: torch.Tensor | None = None, out: torch.Tensor | None = None,
                              stream=None) -> torch.Tensor:
    """cw_suffix_prefill_attn_split: the split-KV path; returns out [total_s, Hq, D] bf16.
    `workspace` (uint8, device) is allocated when not given."""
    if DEBUG_CHECK_COPIES:
        meta.check_device_copies()
    hq, hkv, D = meta.num_q_heads, meta.num_kv_heads, meta.head_dim
    if num_splits is None:
        num_splits = split_count(meta)
    if tuple(q.shape) != (meta.total_rows, hq, D):
        raise ValueError(f"q must be [{meta.total_rows}, {hq}, {D}], got {tuple(q.shape)}")
    if not _cache_shapes_ok(k_cache, v_cache, hkv, D):
        raise ValueError("k_cache and v_cache must both be [num_blocks, Hkv, 16, D]")
    if out is None:
        out = torch.empty_like(q)
    elif tuple(out.shape) != tuple(q.shape):
        raise ValueError("out must have q's shape")
    need = split_workspace_bytes(meta, num_splits)
    if workspace is None:
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=q.device)
    plan_host, plan_dev = meta.split_plan(int(num_splits))
    _check(_lib.cw_suffix_prefill_attn_split(
        _dev(q, torch.bfloat16, "q"), _dev(k_cache, torch.bfloat16, "k_cache"),
        _dev(v_cache, torch.bfloat16, "v_cache"), _dev(meta.bt, torch.int32, "block_table"), meta.bt_stride,
        _dev(meta.cu, torch.int32, "cu_suffix"), _dev(meta.plen, torch.int32, "prefix_len"),
        meta._hp(meta.cu_host), meta._hp(meta.plen_host), meta.batch, hq, hkv, D, BLOCK_SIZE,
        k_cache.shape[0], float(softmax_scale), meta._hp(plan_host), _dev(plan_dev, torch.int32, "plan"),
        _dev(workspace, torch.uint8, "workspace"), workspace.numel(),
        _dev(out, torch.bfloat16, "out"), _stream(stream)))
    return out


def noalloc_scratch_bytes() -> int:
    """Size of the library's built-in scratch for the allocation-free split call."""
    return int(_lib.cw_noalloc_scratch_bytes())


def suffix_prefill_attn_split_noalloc(meta: BatchMeta, q: torch.Tensor, k_cache: torch.Tensor,
                                      v_cache: torch.Tensor, softmax_scale: float, num_splits: int | None = None,
                                      out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """cw_suffix_prefill_attn_split_noalloc: the split path with the library's
    built-in scratch instead of a workspace (the call allocates no device
    memory; `out` must be given by callers that cannot allocate)."""
    if DEBUG_CHECK_COPIES:
        meta.check_device_copies()
    hq, hkv, D = meta.num_q_heads, meta.num_kv_heads, meta.head_dim
    if num_splits is None:
        num_splits = split_count(meta)
    if tuple(q.shape) != (meta.total_rows, hq, D):
        raise ValueError(f"q must be [{meta.total_rows}, {hq}, {D}], got {tuple(q.shape)}")
    if not _cache_shapes_ok(k_cache, v_cache, hkv, D):
        raise ValueError("k_cache and v_cache must both be [num_blocks, Hkv, 16, D]")
    if out is None:
        out = torch.empty_like(q)
    elif tuple(out.shape) != tuple(q.shape):
        raise ValueError("out must have q's shape")
    plan_host, plan_dev = meta.split_plan(int(num_splits))
    _check(_lib.cw_suffix_prefill_attn_split_noalloc(
        _dev(q, torch.bfloat16, "q"), _dev(k_cache, torch.bfloat16, "k_cache"),
        _dev(v_cache, torch.bfloat16, "v_cache"), _dev(meta.bt, torch.int32, "block_table"), meta.bt_stride,
        _dev(meta.cu, torch.int32, "cu_suffix"), _dev(meta.plen, torch.int32, "prefix_len"),
        meta._hp(meta.cu_host), meta._hp(meta.plen_host), meta.batch, hq, hkv, D, BLOCK_SIZE,
        k_cache.shape[0], float(softmax_scale), meta._hp(plan_host), _dev(plan_dev, torch.int32, "plan"),
        _dev(out, torch.bfloat16, "out"), _stream(stream)))
    return out


def lse_merge(partial_o: torch.Tensor, partial_lse: torch.Tensor, out: torch.Tensor | None = None,
              stream=None) -> torch.Tensor:
    """cw_lse_merge: partial_o fp32 [parts, rows, D], partial_lse fp32 [parts, rows]
    -> out bf16 [rows, D]."""
    if partial_o.dim() != 3 or partial_lse.dim() != 2 or tuple(partial_lse.shape) != tuple(partial_o.shape[:2]):
        raise ValueError("partial_o must be [parts, rows, D] and partial_lse [parts, rows]")
    parts, rows, D = partial_o.shape
    if out is None:
        out = torch.empty((rows, D), dtype=torch.bfloat16, device=partial_o.device)
    elif tuple(out.shape) != (rows, D):
        raise ValueError(f"out must be [{rows}, {D}]")
    _check(_lib.cw_lse_merge(_dev(partial_o, torch.float32, "partial_o"), _dev(partial_lse, torch.float32, "partial_lse"),
                             parts, rows, D, _dev(out, torch.bfloat16, "out"), _stream(stream)))
    return out


# ---------------------------------------------------------------- repeated calls
class BatchRunner:
    """Pre-bound calls for running the same kind of batch repeatedly.

    Holds the flattened prompt tokens, host buffers for the block table,
    offsets and plan (pinned when a GPU is present, so their uploads are
    asynchronous), the device copies, and the C entry points with their
    arguments converted once. Each schedule() / upload() / launch call is then
    one ctypes call on cached arguments; the C library still validates every
    call. With fused=True the plan is the fused call's
    (cw_suffix_prefill_append_plan, built for the pool of the caches given to
    bind(), which must come first) and append_attention() runs the append and
    the attention in one launch.
    """

    def __init__(self, prompts, bt_stride: int, num_q_heads: int, num_kv_heads: int, head_dim: int,
                 block_size: int = BLOCK_SIZE, device="cuda", fused: bool = False):
        toks = [_i32_array(p, "tokens") for p in prompts]
        self.batch = B = len(toks)
        self.bt_stride = int(bt_stride)
        self.block_size = int(block_size)
        self.num_q_heads, self.num_kv_heads, self.head_dim = num_q_heads, num_kv_heads, head_dim
        self.tokens = np.ascontiguousarray(np.concatenate(toks), dtype=np.int32)
        self.cu_tokens = np.zeros(B + 1, dtype=np.int64)
        self.cu_tokens[1:] = np.cumsum([len(t) for t in toks])
        pin = torch.cuda.is_available()
        # worst-case plan size: every request with all its prompt as suffix
        max_cu = np.zeros(B + 1, dtype=np.int32)
        max_cu[1:] = np.cumsum(np.diff(self.cu_tokens))
        zero = np.zeros(B, dtype=np.int32)
        self.fused = bool(fused)
        if self.fused:
            words = int(_lib.cw_suffix_prefill_append_plan_words(
                _ptr(max_cu, ctypes.c_int32), _ptr(zero, ctypes.c_int32), self.bt_stride, B, num_q_heads,
                num_kv_heads, head_dim))
        else:
            words = int(_lib.cw_suffix_prefill_plan_words(_ptr(max_cu, ctypes.c_int32), _ptr(zero, ctypes.c_int32),
                                                          B, num_q_heads, num_kv_heads, head_dim, 1))
        if words < 0:
            _check(words)
        # queues of uneven entry counts pad to the longest: leave room for that
        self.plan_capacity = max(2 * words, PLAN_HEADER + PLAN_ENTRY * 256 * 8)
        # One host buffer (pinned when a GPU is present) and one device buffer
        # hold [block table | cu_suffix | prefix_len | plan], so a step uploads
        # its schedule with a single asynchronous copy. Sections start on
        # 16-byte boundaries (the plan is read as 16-byte entries).
        def up4(n):
            return (n + 3) // 4 * 4
        o_bt, o_cu = 0, up4(B * bt_stride)
        o_pl = o_cu + up4(B + 1)
        o_plan = o_pl + up4(B)
        total = o_plan + self.plan_capacity
        self._host = torch.empty(total, dtype=torch.int32, pin_memory=pin)
        h = self._host.numpy()
        self.bt_host = h[o_bt:o_bt + B * bt_stride].reshape(B, bt_stride)
        self.cu_host = h[o_cu:o_cu + B + 1]
        self.plen_host = h[o_pl:o_pl + B]
        self.plan_host = h[o_plan:o_plan + self.plan_capacity]
        self._o_plan = o_plan
        self.plan_words = 0
        self.device = device
        self._dev = torch.empty(total, dtype=torch.int32, device=device)
        self.bt = self._dev[o_bt:o_bt + B * bt_stride].view(B, bt_stride)
        self.cu = self._dev[o_cu:o_cu + B + 1]
        self.plen = self._dev[o_pl:o_pl + B]
        self.plan = self._dev[o_plan:o_plan + self.plan_capacity]
        p32 = lambda a: _ptr(a, ctypes.c_int32)
        self._p = {"tok": p32(self.tokens), "cut": _ptr(self.cu_tokens, ctypes.c_int64), "bt": p32(self.bt_host),
                   "cu": p32(self.cu_host), "pl": p32(self.plen_host), "plan": p32(self.plan_host)}
        self._append_args = None
        self._attn_args = None
        self._fused_args = None
        self._num_blocks = None

    @property
    def total_rows(self) -> int:
        return int(self.cu_host[-1])

    def _plan(self) -> None:
        p = self._p
        if self.fused:
            if self._num_blocks is None:
                raise RuntimeError("a fused runner needs bind() before its first schedule")
            _check(_lib.cw_suffix_prefill_append_plan(p["cu"], p["pl"], p["bt"], self.bt_stride, self.batch,
                                                      self.num_q_heads, self.num_kv_heads, self.head_dim,
                                                      self._num_blocks, p["plan"], self.plan_capacity))
            self.plan_words = int(self.plan_host[HDR_TABLE]) + 2 * self.batch * self.bt_stride
            return
        _check(_lib.cw_suffix_prefill_plan(p["cu"], p["pl"], self.batch, self.num_q_heads, self.num_kv_heads,
                                           self.head_dim, 1, p["plan"], self.plan_capacity))
        self.plan_words = PLAN_HEADER + PLAN_ENTRY * int(self.plan_host[HDR_ENTRIES])

    def schedule(self, pool: Pool) -> None:
        """cw_schedule_batch into the host buffers, then the attention plan."""
        p = self._p
        _check(_lib.cw_schedule_batch(pool.handle, p["tok"], p["cut"], self.batch, self.block_size, self.bt_stride,
                                      p["bt"], p["pl"], p["cu"]))
        self._plan()

    def set_schedule(self, block_table, prefix_len, cu_suffix) -> None:
        """Use a given schedule instead of cw_schedule_batch (fixed-depth batches)."""
        self.bt_host[...] = block_table
        self.plen_host[...] = prefix_len
        self.cu_host[...] = cu_suffix
        self._plan()

    def release(self, pool: Pool) -> None:
        p = self._p
        _check(_lib.cw_release_batch(pool.handle, p["bt"], self.bt_stride, p["pl"], p["cu"], self.batch,
                                     self.block_size))

    def upload(self) -> None:
        """One asynchronous copy of the host schedule to the device buffer (current stream)."""
        n = self._o_plan + self.plan_words
        self._dev[:n].copy_(self._host[:n], non_blocking=True)

    def bind(self, q, k_new, v_new, k_cache, v_cache, out, softmax_scale: float, stream=None) -> None:
        """Fixes the tensors of the device calls (checked once here)."""
        hq, hkv, D = self.num_q_heads, self.num_kv_heads, self.head_dim
        for name, t, dt in (("q", q, torch.bfloat16), ("k_new", k_new, torch.bfloat16),
                            ("v_new", v_new, torch.bfloat16), ("k_cache", k_cache, torch.bfloat16),
                            ("v_cache", v_cache, torch.bfloat16), ("out", out, torch.bfloat16)):
            _dev(t, dt, name)
        if not _cache_shapes_ok(k_cache, v_cache, hkv, D):
            raise ValueError("k_cache and v_cache must both be [num_blocks, Hkv, 16, D]")
        self._tensors = (q, k_new, v_new, k_cache, v_cache, out)
        s = _stream(stream)
        p = self._p
        self._append_args = [k_new.data_ptr(), v_new.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                             self.bt.data_ptr(), self.bt_stride, self.cu.data_ptr(), self.plen.data_ptr(),
                             p["cu"], p["pl"], self.batch, hkv, D, BLOCK_SIZE, k_cache.shape[0], s]
        self._attn_args = [q.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(), self.bt.data_ptr(), self.bt_stride,
                           self.cu.data_ptr(), self.plen.data_ptr(), p["cu"], p["pl"], self.batch, hq, hkv, D,
                           BLOCK_SIZE, k_cache.shape[0], float(softmax_scale), p["plan"], self.plan.data_ptr(),
                           out.data_ptr(), s]
        self._fused_args = [q.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), k_cache.data_ptr(), v_cache.data_ptr(),
                            p["bt"], self.bt_stride, p["cu"], p["pl"], self.batch, hq, hkv, D, BLOCK_SIZE,
                            k_cache.shape[0], float(softmax_scale), p["plan"], self.plan.data_ptr(), out.data_ptr(),
                            s]
        self._num_blocks = int(k_cache.shape[0])
        self._rows = (q.shape[0], k_new.shape[0], v_new.shape[0], out.shape[0])

    def check_device_copies(self) -> None:
        """Checks that the uploaded schedule equals the host one (synchronises)."""
        n = self.plan_words
        _check_copies((("block_table", self.bt, self.bt_host), ("cu_suffix", self.cu, self.cu_host),
                       ("prefix_len", self.plen, self.plen_host), ("plan", self.plan[:n], self.plan_host[:n])))

    def kv_append(self) -> None:
        if any(n != self.total_rows for n in self._rows):
            raise ValueError("bound tensors do not match the scheduled suffix rows")
        if DEBUG_CHECK_COPIES:
            self.check_device_copies()
        _check(_lib.cw_kv_append(*self._append_args))

    def attention(self) -> None:
        if self.fused:
            raise RuntimeError("a fused runner's plan is for append_attention()")
        if any(n != self.total_rows for n in self._rows):
            raise ValueError("bound tensors do not match the scheduled suffix rows")
        if DEBUG_CHECK_COPIES:
            self.check_device_copies()
        _check(_lib.cw_suffix_prefill_attn(*self._attn_args))

    def append_attention(self) -> None:
        """cw_suffix_prefill_append_attn: the append and the attention in one launch."""
        if not self.fused:
            raise RuntimeError("append_attention() needs a runner built with fused=True")
        if any(n != self.total_rows for n in self._rows):
            raise ValueError("bound tensors do not match the scheduled suffix rows")
        if DEBUG_CHECK_COPIES:
            self.check_device_copies()
        _check(_lib.cw_suffix_prefill_append_attn(*self._fused_args))


# ---------------------------------------------------------------- measurement aid
def probe_mfma_bf16_flops(iters: int, workgroups: int) -> int:
    """FLOPs of one cw_probe_mfma_bf16 call."""
    n = int(_lib.cw_probe_mfma_bf16_flops(int(iters), int(workgroups)))
    if n < 0:
        raise ValueError("iters and workgroups must be >= 1")
    return n


def probe_mfma_bf16(operands: torch.Tensor, sink: torch.Tensor, iters: int, workgroups: int, stream=None) -> None:
    """cw_probe_mfma_bf16: back-to-back bf16 MFMA work on fragments of `operands`
    (bf16, a multiple of 512 values); `sink` (float32) receives one value per
    thread and must hold workgroups * 512. Not a step of the path: it measures
    the matrix rate the card sustains on data of a given distribution."""
    if sink.numel() < int(workgroups) * 512:
        raise ValueError(f"sink must hold {int(workgroups) * 512} floats")
    _check(_lib.cw_probe_mfma_bf16(_dev(operands, torch.bfloat16, "operands"), operands.numel() * 2,
                                   _dev(sink, torch.float32, "sink"), int(iters), int(workgroups),
                                   _stream(stream)))
