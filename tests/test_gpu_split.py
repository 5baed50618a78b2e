"""GPU parity of the split-KV attention path and the log-sum-exp merge against
the fp64 oracle (same bars as the plain attention: max-abs <= 2e-2, mean-abs
<= 2e-3 against the unrounded fp64 result)."""
import numpy as np
import pytest
import torch

from oracle import attention as OA
from paper_2606_19667_amd import batch as B
from paper_2606_19667_amd import cw
from paper_2606_19667_amd import workload as W

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-2
MEAN_ABS = 2e-3


def _say(msg):
    print(msg, flush=True)


def _check(got, expect, what):
    d = np.abs(got.astype(np.float64) - expect)
    mx, mean = float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0
    _say(f"{what}: max_abs={mx:.3e} mean_abs={mean:.3e} n={d.size}")
    assert np.isfinite(got).all(), what
    assert mx <= MAX_ABS and mean <= MEAN_ABS, (what, mx, mean)


def _run_split(db, splits):
    cw.kv_append(db.meta, db.k_new, db.v_new, db.k_cache, db.v_cache)
    out = cw.suffix_prefill_attn_split(db.meta, db.q, db.k_cache, db.v_cache, db.scale, num_splits=splits)
    torch.cuda.synchronize()
    return out


def _compare(db, out, requests=None, sample=False):
    outs, exps = [], []
    rng = np.random.default_rng(0)
    for r in (range(db.workload.batch) if requests is None else requests):
        c0, c1 = int(db.sched.cu_suffix[r]), int(db.sched.cu_suffix[r + 1])
        P = int(db.sched.prefix_len[r])
        if sample:
            rows = sorted(set([0, c1 - c0 - 1] + list(rng.integers(0, c1 - c0, size=64))))
            exps.append(OA.suffix_prefill_rows(db.q_host[r], db.logical_k[r], db.logical_v[r], P, db.scale, rows))
            outs.append(out[c0:c1][torch.as_tensor(rows, device=out.device)].float().cpu().numpy())
        else:
            exps.append(OA.suffix_prefill_attention(db.q_host[r], db.logical_k[r], db.logical_v[r], P, db.scale))
            outs.append(out[c0:c1].float().cpu().numpy())
    return np.concatenate(outs), np.concatenate(exps)


@pytest.mark.parametrize("parts,rows,d", [(1, 100, 128), (3, 777, 128), (5, 64, 64), (2, 33, 8)])
def test_lse_merge_matches_oracle(parts, rows, d):
    g = torch.Generator().manual_seed(parts * 1000 + rows + d)
    o = torch.randn((parts, rows, d), generator=g, dtype=torch.float32)
    lse = (torch.rand((parts, rows), generator=g) * 60 - 30).float()
    drop = torch.rand((parts, rows), generator=g) < 0.3
    lse[drop] = -float("inf")
    lse[:, 0] = -float("inf")                       # a row with no keys at all
    if parts > 1:
        lse[0, 1] = 200.0                           # one dominant part
    expect = OA.lse_merge(o.numpy(), lse.numpy())
    got = cw.lse_merge(o.cuda(), lse.cuda())
    torch.cuda.synchronize()
    got = got.float().cpu().numpy()
    assert (got[0] == 0).all()
    _check(got, expect, f"lse_merge parts={parts} rows={rows} d={d}")


@pytest.mark.parametrize("splits", [1, 2, 4, 7])
def test_split_question_only(splits):
    w = W.question_only()
    _say(f"split attention {w.name} splits={splits}")
    db = B.materialize(w)
    _check(*_compare(db, _run_split(db, splits)), f"{w.name} splits={splits}")
    torch.cuda.empty_cache()


def _ragged(hq, hkv, D, S, P, seed):
    prompts = [W.Prompt(uid=i, segments=[(W.SEG_QUESTION_BASE + i, p + s)]) for i, (s, p) in enumerate(zip(S, P))]
    return W.Workload(f"ragged-{hq}q{hkv}kv-d{D}", hq, hkv, D, 16, prompts, seed=seed, prefix_lens=list(P),
                      extra_blocks=5)


@pytest.mark.parametrize("hq,hkv,D,splits", [(4, 4, 64, 3), (32, 8, 128, 3), (16, 1, 64, 5), (64, 8, 128, 64)])
def test_split_ragged(hq, hkv, D, splits):
    S = [1, 15, 16, 17, 600, 0, 33, 129]
    P = [0, 16, 48, 0, 1024, 32, 1008, 64]
    w = _ragged(hq, hkv, D, S, P, seed=hq + D)
    _say(f"split attention {w.name} splits={splits}")
    db = B.materialize(w)
    _check(*_compare(db, _run_split(db, splits)), f"{w.name} splits={splits}")
    torch.cuda.empty_cache()


def test_split_trace_batch():
    w = W.llama8b_trace_batch(seed=2, batch=4, warmup=24)
    db = B.materialize(w)
    _check(*_compare(db, _run_split(db, 2)), f"{w.name} splits=2")
    torch.cuda.empty_cache()


def test_split_long_context_sampled():
    w = W.long_context("high")
    db = B.materialize(w, keep_host=[0, w.batch - 1], gen_device="cuda")
    _check(*_compare(db, _run_split(db, 8), requests=[0, w.batch - 1], sample=True), f"{w.name} splits=8 (sampled)")
    del db
    torch.cuda.empty_cache()
