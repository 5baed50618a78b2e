"""GPU parity of the fused suffix QKV projection + rotary embedding + KV append.

cw_qkv_rope_append runs through the C ABI on seeded synthetic inputs and is
compared with the fp64 oracle (oracle.projection for q/k/v, oracle.paged for
where k and v land in the cache):

* every output element within |got - exp| <= 2^-8 |exp| + 1e-3. The kernel
  rounds each result once to bf16 (half an ulp: 2^-9 relative); fp32
  accumulation of `hidden` exact bf16 products with random signs adds about
  sqrt(hidden) 2^-24 |y| (< 1e-5 at hidden 8192), the fp32 cos/sin table
  another 2^-24 relative. The bound leaves 2x on the rounding term and 100x
  on the rest.
* every cache element that is not a suffix slot keeps its bits exactly;
  suffix slots whose block id lies outside the pool are not written.

Small cases compare everything; the model-sized batches compare sampled rows
(first / last row of every request and random ones) plus the untouched bytes
of the whole cache.
"""
import math

import numpy as np
import pytest
import torch

from oracle import paged as OP
from oracle import projection as PR
from paper_2606_19667_amd import batch as B
from paper_2606_19667_amd import cw, inputs
from paper_2606_19667_amd import workload as W

pytestmark = pytest.mark.gpu

REL = 2.0 ** -8
ABS = 1e-3
BS = 16


def _say(msg):
    print(msg, flush=True)


def _bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def _f64(t):
    return t.float().cpu().numpy().astype(np.float64)


def _close(got, exp, what):
    got = np.asarray(got, np.float64)
    err = np.abs(got - exp)
    bound = REL * np.abs(exp) + ABS
    worst = float((err - bound).max()) if err.size else -1.0
    _say(f"{what}: n={err.size} max_abs={float(err.max()) if err.size else 0:.3e} "
         f"mean_abs={float(err.mean()) if err.size else 0:.3e} worst_margin={worst:.3e}")
    assert np.isfinite(got).all(), what
    assert (err <= bound).all(), (what, worst)


def _image(cache, new, bt, cu, plen, layout):
    """Expected cache image; slots whose block id is outside the pool are dropped
    (written to a padding block that is cut off again)."""
    nb = cache.shape[0]
    bt2 = np.where((bt >= 0) & (bt < nb), bt, nb)
    ext = np.concatenate([cache, np.zeros_like(cache[:1])])
    return OP.kv_append_image(ext, new, bt2, cu, plen, BS, layout)[:nb]


class Case:
    """A ragged batch, its inputs and the library's outputs."""

    def __init__(self, name, hq, hkv, D, hidden, bt, cu, plen, num_blocks, seed, bias=True, base=500000.0):
        self.name, self.hq, self.hkv, self.D, self.hidden = name, hq, hkv, D, hidden
        self.bt = np.asarray(bt, np.int32)
        self.cu = np.asarray(cu, np.int32)
        self.plen = np.asarray(plen, np.int32)
        self.base = base
        T = int(self.cu[-1])
        nf = (hq + 2 * hkv) * D
        self.x = inputs.normal_bf16((seed, 101), (T, hidden))
        self.w = inputs.scaled_normal_bf16((seed, 102), (nf, hidden), hidden ** -0.5)
        self.b = inputs.scaled_normal_bf16((seed, 103), (nf,), 0.5) if bias else None
        self.k0 = inputs.normal_bf16((seed, 104), (num_blocks, hkv, BS, D))
        self.v0 = inputs.normal_bf16((seed, 105), (num_blocks, hkv, BS, D))
        self.pos = PR.suffix_positions(self.cu, self.plen)

    def run(self):
        meta = cw.BatchMeta(self.bt, self.cu, self.plen, self.hq, self.hkv, self.D)
        n_pos = int(self.pos.max()) + 1 if self.pos.size else 1
        rope = torch.from_numpy(cw.rope_table(n_pos, self.D, self.base)).cuda()
        self.kc, self.vc = self.k0.cuda(), self.v0.cuda()
        _say(f"qkv_rope_append {self.name}: T={int(self.cu[-1])} hidden={self.hidden} "
             f"Hq={self.hq} Hkv={self.hkv} D={self.D} bias={self.b is not None}")
        q = cw.qkv_rope_append(meta, self.x.cuda(), self.w.cuda(), rope, self.kc, self.vc,
                               bias=None if self.b is None else self.b.cuda())
        torch.cuda.synchronize()
        self.q = q
        return self

    def expected(self, rows):
        rows = np.asarray(rows, np.int64)
        return PR.qkv_rope(self.x[torch.as_tensor(rows)], self.w, self.pos[rows], self.hq, self.hkv, self.D,
                           self.base, self.b)

    def written_mask(self):
        T = int(self.cu[-1])
        ones = np.ones((T, self.hkv, self.D), bool)
        mk = _image(np.zeros(self.k0.shape, bool), ones, self.bt, self.cu, self.plen, "slot_d")
        mv = _image(np.zeros(self.v0.shape, bool), ones, self.bt, self.cu, self.plen, "slot_d")
        return mk, mv

    def check_untouched(self):
        mk, mv = self.written_mask()
        assert np.array_equal(_bits(self.kc)[~mk], _bits(self.k0)[~mk]), self.name
        assert np.array_equal(_bits(self.vc)[~mv], _bits(self.v0)[~mv]), self.name
        return mk, mv

    def check_full(self):
        T = int(self.cu[-1])
        q, k, v = self.expected(np.arange(T))
        _close(_f64(self.q), q, self.name + " q")
        mk, mv = self.check_untouched()
        ek = _image(_f64(self.k0), k, self.bt, self.cu, self.plen, "slot_d")
        ev = _image(_f64(self.v0), v, self.bt, self.cu, self.plen, "slot_d")
        _close(_f64(self.kc)[mk], ek[mk], self.name + " k cache")
        _close(_f64(self.vc)[mv], ev[mv], self.name + " v cache")

    def check_sampled(self, seed=0, n_random=64):
        rng = np.random.default_rng(seed)
        rows = set()
        for r in range(len(self.plen)):
            c0, c1 = int(self.cu[r]), int(self.cu[r + 1])
            if c1 > c0:
                rows.update({c0, c1 - 1})
        T = int(self.cu[-1])
        rows.update(int(t) for t in rng.integers(0, T, size=n_random))
        rows = np.array(sorted(rows))
        q, k, v = self.expected(rows)
        _close(_f64(self.q[torch.as_tensor(rows, device=self.q.device)]), q, self.name + " q (sampled rows)")
        self.check_untouched()
        kc, vc = _f64(self.kc), _f64(self.vc)
        gk, gv, ek, ev = [], [], [], []
        req = np.searchsorted(self.cu, rows, side="right") - 1
        for i, (t, r) in enumerate(zip(rows, req)):
            p = int(self.pos[t])
            blk = int(self.bt[r, p // BS])
            if 0 <= blk < kc.shape[0]:
                gk.append(kc[blk, :, p % BS, :])
                gv.append(vc[blk, :, p % BS, :])
                ek.append(k[i])
                ev.append(v[i])
        _close(np.stack(gk), np.stack(ek), self.name + " k cache (sampled rows)")
        _close(np.stack(gv), np.stack(ev), self.name + " v cache (sampled rows)")


def _ragged(name, hq, hkv, D, hidden, plen, slen, seed, holes=(), spare=3, **kw):
    """Blocks of every request drawn from a random permutation of the pool;
    holes: (request, logical block, id) entries overwritten afterwards."""
    rng = inputs.rng((seed, 106))
    nblk = [math.ceil((p + s) / BS) for p, s in zip(plen, slen)]
    nb = sum(nblk) + spare
    perm = rng.permutation(nb)
    bt = np.full((len(plen), max(1, max(nblk))), -1, np.int32)
    o = 0
    for r, n in enumerate(nblk):
        bt[r, :n] = perm[o:o + n]
        o += n
    for r, j, v in holes:
        bt[r, j] = v
    cu = np.concatenate([[0], np.cumsum(slen)]).astype(np.int32)
    return Case(name, hq, hkv, D, hidden, bt, cu, plen, nb, seed, **kw)


SMALL = [
    # tiny shape: 6 heads of 64 = 384 features (a partial feature tile), one request
    ("tiny-d64", 4, 1, 64, 256, [64], [32], {}),
    # several token tiles with a ragged tail, empty and one-row requests, bias off
    ("ragged-d128", 8, 2, 128, 512, [0, 48, 16, 0, 320, 32], [300, 0, 1, 17, 129, 211], {"bias": False}),
    # group 1, 3 heads = 384 features (partial tile), one and two hidden steps
    ("g1-h32", 1, 1, 128, 32, [0, 16], [40, 230], {}),
    ("g1-h64", 1, 1, 128, 64, [32, 16], [70, 190], {"base": 10000.0}),
    # three hidden steps, D = 64 with many heads
    ("d64-h96", 16, 4, 64, 96, [16, 0], [260, 5], {}),
    # Qwen2.5-7B-shaped heads (28 Q / 4 KV, hidden 3584, bias)
    ("qwen7b-heads", 28, 4, 128, 3584, [832, 96], [97, 250], {"base": 1e6}),
]


@pytest.mark.parametrize("name,hq,hkv,D,hidden,plen,slen,kw", SMALL, ids=[c[0] for c in SMALL])
def test_qkv_rope_append_matches_oracle(name, hq, hkv, D, hidden, plen, slen, kw):
    _ragged(name, hq, hkv, D, hidden, plen, slen, seed=7, **kw).run().check_full()


def test_blocks_outside_the_pool_are_skipped():
    # request 0's second block is -1, request 1's first is past the pool: nothing lands there
    c = _ragged("holes", 8, 2, 128, 128, [0, 16], [40, 33], seed=9, holes=[(0, 1, -1), (1, 1, 10 ** 6)])
    c.run().check_full()
    assert c.written_mask()[0].sum() == (40 - 16 + 33 - 16) * 2 * 128


def test_empty_batch_writes_nothing():
    c = _ragged("empty", 8, 2, 128, 128, [16, 32], [0, 0], seed=3)
    c.run()
    assert c.q.shape == (0, 8, 128)
    assert np.array_equal(_bits(c.kc), _bits(c.k0)) and np.array_equal(_bits(c.vc), _bits(c.v0))


def test_position_zero_query_is_the_plain_projection():
    # at p = 0 the rotation is the identity: q and k equal y rounded to bf16
    c = _ragged("p0", 4, 1, 64, 64, [0], [1], seed=4)
    c.run()
    y = PR.project(c.x, c.w, c.b)[0]
    _close(_f64(c.q)[0].reshape(-1), y[:4 * 64], "p0 q = y")


def test_llama8b_single_full_size():
    w = W.llama8b_single()
    s = B.schedule(w)
    c = Case(w.name, 32, 8, 128, 4096, s.block_table, s.cu_suffix, s.prefix_len, s.num_blocks, seed=11)
    c.run().check_full()


def test_llama8b_trace_batch16_sampled():
    w = W.llama8b_trace_batch(seed=0, batch=16)
    s = B.schedule(w)
    c = Case(w.name, 32, 8, 128, 4096, s.block_table, s.cu_suffix, s.prefix_len, s.num_blocks, seed=12)
    c.run().check_sampled()


def test_llama70b_long_sampled():
    w = W.long_context("high", batch=3)
    s = B.schedule(w)
    c = Case(w.name, 64, 8, 128, 8192, s.block_table, s.cu_suffix, s.prefix_len, s.num_blocks, seed=13,
             bias=False)
    c.run().check_sampled()
