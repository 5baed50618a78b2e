"""Reference for the integer side of prefix caching: block hashes, block pool,
prefix lookup and the KV-cache image after an append.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Paper Sec. 2.1 (with Fig. 1): the serving engine keeps KV memory in fixed-size
token blocks (16 tokens in the measured runs); each block is hashed together
with its prefix history, so a request reuses the longest leading run of blocks
whose chained hashes are already stored, and a mismatch at an early block ends
all later reuse. Sec. 3.4: the engine owns residency and evicts blocks by
itself. The paper names no hash function; the reading taken here is XXH64 (the
published xxHash 64-bit algorithm) over the block's token IDs as little-endian
int32, keyed by the previous block's hash as the seed:

    h_b = XXH64(LE32(tok[16b]) .. LE32(tok[16b + 15]), seed = h_{b-1}),  h_{-1} = 0

Only full blocks get a hash; a trailing partial block never matches.
"""
from __future__ import annotations

import struct

import numpy as np

_M64 = (1 << 64) - 1
_P1 = 0x9E3779B185EBCA87
_P2 = 0xC2B2AE3D27D4EB4F
_P3 = 0x165667B19E3779F9
_P4 = 0x85EBCA77C2B2AE63
_P5 = 0x27D4EB2F165667C5


def _rotl(x: int, r: int) -> int:
    return ((x << r) | (x >> (64 - r))) & _M64


def _round(acc: int, lane: int) -> int:
    acc = (acc + lane * _P2) & _M64
    return (_rotl(acc, 31) * _P1) & _M64


def _merge(acc: int, val: int) -> int:
    acc ^= _round(0, val)
    return (acc * _P1 + _P4) & _M64


def xxh64(data: bytes, seed: int = 0) -> int:
    """XXH64 of `data` with a 64-bit seed, written from the published algorithm
    (four-lane 32-byte stripes, then 8-, 4- and 1-byte tails, then avalanche)."""
    n = len(data)
    i = 0
    seed &= _M64
    if n >= 32:
        v1 = (seed + _P1 + _P2) & _M64
        v2 = (seed + _P2) & _M64
        v3 = seed
        v4 = (seed - _P1) & _M64
        while i + 32 <= n:
            a, b, c, d = struct.unpack_from("<4Q", data, i)
            v1 = _round(v1, a)
            v2 = _round(v2, b)
            v3 = _round(v3, c)
            v4 = _round(v4, d)
            i += 32
        acc = (_rotl(v1, 1) + _rotl(v2, 7) + _rotl(v3, 12) + _rotl(v4, 18)) & _M64
        for lane in (v1, v2, v3, v4):
            acc = _merge(acc, lane)
    else:
        acc = (seed + _P5) & _M64
    acc = (acc + n) & _M64
    while i + 8 <= n:
        (w,) = struct.unpack_from("<Q", data, i)
        acc ^= _round(0, w)
        acc = (_rotl(acc, 27) * _P1 + _P4) & _M64
        i += 8
    if i + 4 <= n:
        (w,) = struct.unpack_from("<I", data, i)
        acc ^= (w * _P1) & _M64
        acc = (_rotl(acc, 23) * _P2 + _P3) & _M64
        i += 4
    while i < n:
        acc ^= (data[i] * _P5) & _M64
        acc = (_rotl(acc, 11) * _P1) & _M64
        i += 1
    acc ^= acc >> 33
    acc = (acc * _P2) & _M64
    acc ^= acc >> 29
    acc = (acc * _P3) & _M64
    acc ^= acc >> 32
    return acc


def chain_block_hashes(tokens, block_size: int = 16) -> list:
    """Chained hashes of the full blocks of one prompt (list of Python ints)."""
    toks = [int(t) for t in tokens]
    out = []
    h = 0
    for b in range(len(toks) // block_size):
        chunk = toks[b * block_size:(b + 1) * block_size]
        h = xxh64(struct.pack(f"<{block_size}i", *chunk), h)
        out.append(h)
    return out


class PoolSim:
    """Block pool with chained-hash lookup, reference counts and LRU reuse.

    State: per block a reference count and an optional stored hash; a map from
    stored hash to block; a free queue holding exactly the blocks whose count is
    zero, in the order they will be handed out.

    * prefix_match: longest leading run of hashes present in the map (at most
      `max_match`); each matched block gains a reference (leaving the free queue
      if its count was zero).
    * alloc: hands out blocks from the front of the free queue; a block handed
      out forgets its stored hash (that is eviction). Too few free blocks: no
      change, error.
    * commit: stores hash -> block for held blocks (a block may store one hash
      only, and may not be listed with two); if the hash is already stored for
      another block the map keeps the first one.
    * release: drops one reference per listed block; blocks reaching zero join
      the back of the free queue in reverse listing order, so the tail of a
      released sequence is reused before its head.
    Invalid calls raise ValueError and change nothing.
    """

    def __init__(self, num_blocks: int, free_order=None):
        self.num_blocks = int(num_blocks)
        order = list(range(num_blocks)) if free_order is None else [int(b) for b in free_order]
        if sorted(order) != list(range(num_blocks)):
            raise ValueError("free_order must be a permutation of the block IDs")
        self.ref = [0] * num_blocks
        self.hash_of = [None] * num_blocks
        self.table = {}
        self.free = list(order)

    def prefix_match(self, hashes, max_match: int):
        ids = []
        for h in list(hashes)[:max(0, max_match)]:
            b = self.table.get(int(h))
            if b is None:
                break
            ids.append(b)
        for b in ids:
            if self.ref[b] == 0:
                self.free.remove(b)
            self.ref[b] += 1
        return ids

    def alloc(self, n: int):
        if n < 0 or n > len(self.free):
            raise ValueError("not enough free blocks")
        ids = self.free[:n]
        del self.free[:n]
        for b in ids:
            if self.hash_of[b] is not None:
                del self.table[self.hash_of[b]]
                self.hash_of[b] = None
            self.ref[b] = 1
        return ids

    def commit(self, hashes, ids):
        hashes = [int(h) for h in hashes]
        ids = [int(b) for b in ids]
        pending = {}
        for h, b in zip(hashes, ids):
            if not (0 <= b < self.num_blocks) or self.ref[b] == 0:
                raise ValueError("commit of a block that is not held")
            if self.hash_of[b] is not None and self.hash_of[b] != h:
                raise ValueError("block already holds another hash")
            if pending.setdefault(b, h) != h:
                raise ValueError("block listed with two hashes")
        for h, b in zip(hashes, ids):
            if self.hash_of[b] is not None:
                continue
            if h in self.table:
                continue
            self.table[h] = b
            self.hash_of[b] = h

    def release(self, ids):
        ids = [int(b) for b in ids]
        counts = {}
        for b in ids:
            if not (0 <= b < self.num_blocks):
                raise ValueError("block ID out of range")
            counts[b] = counts.get(b, 0) + 1
        for b, c in counts.items():
            if c > self.ref[b]:
                raise ValueError("release of a block that is not held")
        for b in reversed(ids):
            self.ref[b] -= 1
            if self.ref[b] == 0:
                self.free.append(b)


def kv_append_image(cache, new, block_table, cu_suffix, prefix_len, block_size: int = 16,
                    layout: str = "slot_d"):
    """Expected cache after writing each request's suffix K (or V) into its blocks.

    Paper Sec. 2.1: the K/V of a prompt live in fixed-size blocks named by a
    per-request block table; after the prefix match only the suffix tokens'
    K/V are computed and written. Token t of request r (P_r <= t < P_r + S_r)
    lands in block block_table[r, t // bs] at slot t % bs; every other
    element keeps its value.

    A table entry outside [0, NB) names no block of the pool (the paper's
    engine never produces one; the reading taken for a corrupted table is that
    the write is dropped): those tokens change nothing.

    layout "slot_d": cache is [NB, Hkv, bs, D] (the K cache);
    layout "d_slot": cache is [NB, Hkv, D, bs], each block stored transposed
    (the V cache). new: [total_s, Hkv, D]; block_table: [B, stride] int;
    cu_suffix: [B + 1]; prefix_len: [B]. Bits are copied, never converted.
    """
    if layout not in ("slot_d", "d_slot"):
        raise ValueError(f"unknown layout {layout!r}")
    out = np.array(cache, copy=True)
    nb = out.shape[0]
    new = np.asarray(new)
    bt = np.asarray(block_table)
    for r in range(len(prefix_len)):
        p = int(prefix_len[r])
        s = int(cu_suffix[r + 1]) - int(cu_suffix[r])
        t = np.arange(p, p + s)
        blocks = bt[r, t // block_size].astype(np.int64)
        keep = (blocks >= 0) & (blocks < nb)
        t, blocks = t[keep], blocks[keep]
        slots = t % block_size
        rows = new[int(cu_suffix[r]) + (t - p)]          # [s, Hkv, D]
        if layout == "slot_d":
            out[blocks, :, slots, :] = rows
        else:
            out[blocks, :, :, slots] = rows
    return out


def kv_append_image_loops(cache, new, block_table, cu_suffix, prefix_len, block_size: int = 16,
                          layout: str = "slot_d"):
    """The same scatter as `kv_append_image`, one element at a time."""
    out = np.array(cache, copy=True)
    D = np.asarray(new).shape[2]
    for r in range(len(prefix_len)):
        p = int(prefix_len[r])
        s = int(cu_suffix[r + 1]) - int(cu_suffix[r])
        for i in range(s):
            t = p + i
            blk = int(block_table[r][t // block_size])
            if not 0 <= blk < out.shape[0]:
                continue
            for g in range(out.shape[1]):
                for d in range(D):
                    val = new[int(cu_suffix[r]) + i, g, d]
                    if layout == "slot_d":
                        out[blk, g, t % block_size, d] = val
                    else:
                        out[blk, g, d, t % block_size] = val
    return out


def zero_out_of_pool_blocks(x, block_row, num_blocks: int, block_size: int = 16):
    """Logical K (or V) rows [L, Hkv, D] of one request as attention reads them
    through its block-table row: the rows of logical block b whose table entry
    block_row[b] lies outside [0, num_blocks) are zeros (the reading taken for a
    table entry that names no block of the pool: the paper's engine never
    produces one). Every other row is unchanged. Returns a float64 copy."""
    if hasattr(x, "detach"):
        x = x.detach().to("cpu").double().numpy()
    out = np.array(x, dtype=np.float64, copy=True)
    L = out.shape[0]
    for b in range((L + block_size - 1) // block_size):
        blk = int(block_row[b])
        if not 0 <= blk < num_blocks:
            out[b * block_size:min(L, (b + 1) * block_size)] = 0.0
    return out
