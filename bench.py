"""Throughput of suffix prefill over paged cached prefixes on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

Workload (default): a batch of 16 concurrent requests from a synthetic RAG
trace (pool of 200 chunks of 256 tokens, top-5 retrieval, 3 of 5 chunks shared
with the previous query, evidence ordered by the greedy knowledge-tree walk,
64-token instruction and question, 1408-token prompts) with Llama-3-8B-shaped
attention (32 query heads, 8 KV heads, head_dim 128, 16-token blocks, bf16).
The requests' cached depths are whatever the block pool matches after 64
warm-up queries were served.

One step is one pass of the whole path over that batch:
  host   clone the pool state, cw_schedule_batch (chained hashes, prefix match,
         allocation, commit), cw_suffix_prefill_append_plan, async copy of the
         block table / offsets / plan through pinned buffers;
  device cw_suffix_prefill_append_attn: the KV append and the attention of one
         layer in one launch (the same cache image and output as cw_kv_append
         followed by cw_suffix_prefill_attn);
  host   cw_release_batch.
Inputs (Q and the new K/V rows, the cached prefix blocks) are resident in HBM
before timing starts. K steps are timed between two device synchronisations;
the kernel is also timed on its own with HIP events on its stream. The same
steps with the two separate calls are timed too (key separate_calls).

Prints one JSON line. `value` is attention TFLOP/s over the whole step
(algorithmic FLOPs 4 * D * Hq * sum_r (S_r P_r + S_r (S_r + 1) / 2)).
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
SETTLE_S = 0.1              # untimed steps before the warm-up steps (clock settle)


def attention_flops(prefix_len, suffix_len, hq, d) -> int:
    pairs = sum(int(s) * int(p) + int(s) * (int(s) + 1) // 2 for p, s in zip(prefix_len, suffix_len))
    return int(4 * d * hq * pairs)


def attention_bytes(prefix_len, suffix_len, hq, hkv, d) -> int:
    """Algorithmic HBM bytes of one attention launch: Q read and O written once,
    every request's K and V read once (prefix and suffix)."""
    tot = 0
    for p, s in zip(prefix_len, suffix_len):
        p, s = int(p), int(s)
        tot += 2 * s * hq * d * 2 + 2 * (p + s) * hkv * d * 2
    return tot


def append_bytes(suffix_len, hkv, d) -> int:
    """kv_append: read the new K and V rows, write them into the cache."""
    return int(2 * 2 * int(sum(suffix_len)) * hkv * d * 2)


PROFILE = os.path.join(ROOT, "profiles", "attention_llama8b_trace_b16.txt")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2606_19667_amd", "csrc", "cw_kernels.hip")


def counted_traffic(workload: str):
    """HBM bytes per launch of the fused append + attention kernel from the
    committed rocprofv3 FETCH_SIZE / WRITE_SIZE summary (already scaled by the
    copy calibration), or None when that summary is for another workload or an
    older kernel source."""
    import hashlib
    try:
        fields = dict(line.split(": ", 1) for line in open(PROFILE).read().splitlines()
                      if ": " in line and not line.startswith("#"))
        src = hashlib.sha256(open(KERNEL_SOURCE, "rb").read()).hexdigest()[:16]
    except OSError:
        return None
    if workload != "llama8b-trace-b16" or fields.get("kernel_source_sha256_16") != src:
        return None
    return int(fields["append_attention_traffic_bytes"])


def make_workload(name: str, seed: int):
    from paper_2606_19667_amd import workload as W
    if name == "llama8b-trace-b16":
        return W.llama8b_trace_batch(seed=seed)
    if name == "llama8b-single":
        return W.llama8b_single(seed)
    if name.startswith("topk10-f"):
        return W.topk_sweep(float(name[len("topk10-f"):]), seed)
    if name in ("llama70b-long-low", "llama70b-long-high"):
        return W.long_context(name.rsplit("-", 1)[1], seed)
    if name == "tiny":
        return W.tiny_single(seed)
    if name == "llama8b-question-only":
        return W.question_only(seed)
    raise SystemExit(f"unknown workload {name}")


def executed_mfma_flops(cu_suffix, prefix_len, hq: int, hkv: int, D: int) -> int:
    """MFMA FLOPs the attention kernel executes: every entry of the plan runs
    its 64-key steps [kbeg, kend) over all 256 packed rows (QK^T and PV),
    masked keys and padding rows included. Divided by the algorithmic FLOPs
    this is the masked-tile waste factor."""
    from paper_2606_19667_amd import cw
    ents = cw.plan_entries(cw.suffix_prefill_plan(cu_suffix, prefix_len, hq, hkv, D))
    real = ents[:, cw.ENT_R] >= 0
    steps = int((ents[real, cw.ENT_KEND] - ents[real, cw.ENT_KBEG]).astype(np.int64).sum())
    return steps * 256 * 64 * D * 4


def percentiles_us(times_ms):
    t = np.asarray(times_ms, dtype=np.float64) * 1e3
    return {"median": round(float(np.median(t)), 2), "p10": round(float(np.percentile(t, 10)), 2),
            "p90": round(float(np.percentile(t, 90)), 2), "n": int(t.size)}


def timed_calls(fn, stream, n: int, between=None):
    """Per-call durations (ms) of `fn` with HIP events on `stream`; `between`
    runs before each call, outside the timed interval."""
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    for a, b in evs:
        if between is not None:
            between()
        a.record(stream)
        fn()
        b.record(stream)
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in evs]


def host_timing(w, snapshot, stride: int, reps: int = 20):
    """Host side per request, in microseconds: cw_schedule_batch over the batch
    (chained hashes, prefix match, allocation, commit) and the greedy
    knowledge-tree ordering of the trace's queries (libcw's tree)."""
    from paper_2606_19667_amd import cw
    from paper_2606_19667_amd import workload as W
    toks = [p.tokens(w.seed) for p in w.prompts]
    best = float("inf")
    for _ in range(reps):
        pool = snapshot.clone()
        t0 = time.perf_counter()
        cw.schedule_batch(pool, toks, stride, w.block_size)
        best = min(best, time.perf_counter() - t0)
        pool.close()
    res = {"schedule_us_per_request": round(best * 1e6 / w.batch, 2)}
    if w.warmup:
        # The trace's queries through cw_tree_order (greedy) + cw_tree_insert,
        # called with prepared arrays so the figure is the library's cost plus
        # one ctypes call each.
        import ctypes
        qs = [np.asarray(q, dtype=np.int64) for q in W.synthetic_trace(len(w.warmup) + w.batch, seed=w.seed)]
        lib = cw.lib()
        i64p = ctypes.POINTER(ctypes.c_int64)
        outs = [np.zeros(len(q), dtype=np.int64) for q in qs]
        args = [(q.ctypes.data_as(i64p), len(q), o.ctypes.data_as(i64p)) for q, o in zip(qs, outs)]
        depth, probes = ctypes.c_int32(0), ctypes.c_int32(0)
        best = float("inf")
        for _ in range(reps):
            tree = cw.KnowledgeTree()
            h = tree._h
            t0 = time.perf_counter()
            for qp, k, op in args:
                lib.cw_tree_order(h, cw.ORDER_GREEDY, qp, k, op, ctypes.byref(depth), ctypes.byref(probes))
                lib.cw_tree_insert(h, op, k)
            best = min(best, time.perf_counter() - t0)
            tree.close()
        res["ordering_us_per_request"] = round(best * 1e6 / len(qs), 2)
        res["ordering_impl"] = "libcw knowledge tree: cw_tree_order (greedy) + cw_tree_insert per query"
    return res


def ordering_point(seed: int) -> dict:
    """The ordering side on a 200-query trace of the measured workload's
    generator (200 chunks of 256 tokens, top-5, 3 of 5 shared): the
    prefill-saved proxy (cached prompt tokens / prompt tokens) of each
    ordering strategy with an unbounded pool, and of the greedy walk with and
    without stale-path feedback when the pool holds only a few prompts. The
    first 5 queries are warm-up."""
    from paper_2606_19667_amd import replay as R
    from paper_2606_19667_amd import workload as W
    qs = W.synthetic_trace(200, pool_size=200, k=5, shared=3, seed=seed)
    out = {"trace": "200 queries, 200 chunks x 256 tokens, top-5, 3 of 5 shared, window 32; "
                    "first 5 queries are warm-up", "strategies": {}, "tight_pool": {}}
    for s in ("retrieval", "sorted", "recency", "greedy", "exhaustive"):
        out["strategies"][s] = R.replay(qs, s, seed=seed).summary(skip=5)
    for prompts in (4, 8, 16):
        for fb in (False, True):
            rec = R.replay(qs, "greedy", num_blocks=prompts * 88, feedback=fb, seed=seed)
            out["tight_pool"][f"{prompts}_prompts" + ("_feedback" if fb else "")] = rec.summary(skip=5)
    return out


def question_only_point(seed: int, stream):
    """Diagnostic short-suffix point: 16 8B-shaped requests with the whole
    1344-token evidence prefix cached and a 64-token question to prefill.
    Arithmetic intensity is below the ridge, so it is judged by GB/s."""
    import torch
    from paper_2606_19667_amd import batch as B
    from paper_2606_19667_amd import cw
    w = make_workload("llama8b-question-only", seed)
    db = B.materialize(w, device="cuda", keep_host=[])
    cw.kv_append(db.meta, db.k_new, db.v_new, db.k_cache, db.v_cache)
    out = torch.empty_like(db.q)
    fn = lambda: cw.suffix_prefill_attn(db.meta, db.q, db.k_cache, db.v_cache, db.scale, out=out, stream=stream)
    for _ in range(10):
        fn()
    t = percentiles_us(timed_calls(fn, stream, 50))
    S = np.diff(db.sched.cu_suffix)
    P = db.sched.prefix_len
    hq, hkv, D = w.num_q_heads, w.num_kv_heads, w.head_dim
    fl = attention_flops(P, S, hq, D)
    by = attention_bytes(P, S, hq, hkv, D)
    sec = t["median"] * 1e-6
    res = {"workload": w.name, "attention_us": t, "GFLOP": round(fl / 1e9, 3), "algorithmic_MB": round(by / 1e6, 2),
           "achieved_GBps": round(by / sec / 1e9, 1), "frac_hbm": round(by / sec / 1e9 / PEAK_HBM_GBS, 4),
           "achieved_TFLOPs": round(fl / sec / 1e12, 2), "bound": "hbm"}
    # the split-KV path (cw_suffix_prefill_attn_split, merge included)
    res["split"] = {}
    for n in sorted({cw.split_count(db.meta), 2, 4}):
        ws = torch.empty(cw.split_workspace_bytes(db.meta, n), dtype=torch.uint8, device="cuda")
        fs = lambda: cw.suffix_prefill_attn_split(db.meta, db.q, db.k_cache, db.v_cache, db.scale, num_splits=n,
                                                  workspace=ws, out=out, stream=stream)
        for _ in range(10):
            fs()
        ts = percentiles_us(timed_calls(fs, stream, 50))
        sec = ts["median"] * 1e-6
        res["split"][str(n)] = {"attention_us": ts, "achieved_GBps": round(by / sec / 1e9, 1),
                                "frac_hbm": round(by / sec / 1e9 / PEAK_HBM_GBS, 4),
                                "workspace_MB": round(ws.numel() / 1e6, 2)}
        del ws
    res["split_auto"] = cw.split_count(db.meta)
    return res


def config_points(seed: int, stream, names=("llama8b-single", "topk10-f0.0", "topk10-f0.6", "llama70b-long-high",
                                           "llama70b-long-low")) -> dict:
    """Attention time of the other configurations (not the headline): the
    single 8B-shaped request, the top-k sweep at 0 % and 60 % cached blocks and
    the 70B-shaped long-context batch in trie order (high hit) and retrieval
    order (low hit). Each batch is materialised on the GPU, its suffix
    appended, then the attention call is timed with HIP events (median of
    several calls after calls for SETTLE_S seconds, so that the clock has
    settled under this batch's load)."""
    import torch
    from paper_2606_19667_amd import batch as B
    from paper_2606_19667_amd import cw
    out_all = {}
    for name in names:
        w = make_workload(name, seed)
        db = B.materialize(w, device="cuda", keep_host=[], gen_device="cuda")
        cw.kv_append(db.meta, db.k_new, db.v_new, db.k_cache, db.v_cache)
        out = torch.empty_like(db.q)
        S = np.diff(db.sched.cu_suffix)
        P = db.sched.prefix_len
        hq, hkv, D = w.num_q_heads, w.num_kv_heads, w.head_dim
        fl = attention_flops(P, S, hq, D)
        fn = lambda: cw.suffix_prefill_attn(db.meta, db.q, db.k_cache, db.v_cache, db.scale, out=out, stream=stream)
        n = max(3, min(50, int(2e12 / fl)))
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < 3 * SETTLE_S:
            fn()
            torch.cuda.synchronize()
        t = percentiles_us(timed_calls(fn, stream, n))
        sec = t["median"] * 1e-6
        out_all[name] = {"attention_us": t, "GFLOP": round(fl / 1e9, 3),
                         "achieved_TFLOPs": round(fl / sec / 1e12, 2),
                         "frac": round(fl / sec / 1e12 / PEAK_BF16_TFLOPS, 4),
                         "batch": int(S.size), "suffix_tokens": int(S.sum()), "prefix_tokens": int(P.sum())}
        # a batch of fewer tiles than CUs: also the split-KV call (merge
        # included) at the automatic split count
        ns = cw.split_count(db.meta)
        if ns > 1:
            ws = torch.empty(cw.split_workspace_bytes(db.meta, ns), dtype=torch.uint8, device="cuda")
            fs = lambda: cw.suffix_prefill_attn_split(db.meta, db.q, db.k_cache, db.v_cache, db.scale,
                                                      num_splits=ns, workspace=ws, out=out, stream=stream)
            for _ in range(10):
                fs()
            ts = percentiles_us(timed_calls(fs, stream, n))
            out_all[name]["split"] = {"splits": ns, "tiles": int(db.meta.num_tiles), "attention_us": ts,
                                      "frac": round(fl / (ts["median"] * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4)}
            del ws
        del db, out
        torch.cuda.empty_cache()
    return out_all


def mfma_peak_point(seed: int, stream, workgroups: int = 1024, iters: int = 2000) -> dict:
    """The bf16 MFMA rate this card sustains (cw_probe_mfma_bf16: 8 independent
    32x32x16 accumulators per wave, two waves per SIMD, no memory traffic), on
    normal random bf16 fragments like the workload's Q/K/V and on all-zero
    fragments. The power limit lowers the clock more for random operand bits,
    so the first is the ceiling that applies to the attention kernel; the
    roofline above stays priced against the data-sheet 2.5 PFLOP/s."""
    import torch
    from paper_2606_19667_amd import cw, inputs
    n = 4096 * 512
    sink = torch.empty(workgroups * 512, dtype=torch.float32, device="cuda")
    fl = cw.probe_mfma_bf16_flops(iters, workgroups)
    out = {"kernel": "mfma_probe_kernel (v_mfma_f32_32x32x16_bf16, 8 waves per CU)", "GFLOP_per_call": round(fl / 1e9, 2)}
    for name, ops in (("normal_bf16", inputs.normal_bf16((seed, 301), (n,), "cuda")),
                      ("zero", torch.zeros(n, dtype=torch.bfloat16, device="cuda"))):
        fn = lambda: cw.probe_mfma_bf16(ops, sink, iters, workgroups, stream=stream)
        t0 = time.perf_counter()
        while time.perf_counter() - t0 < SETTLE_S:
            fn()
            torch.cuda.synchronize()
        t = percentiles_us(timed_calls(fn, stream, 10))
        out[name] = {"us": t, "TFLOPs": round(fl / (t["median"] * 1e-6) / 1e12, 1)}
    return out


def qkv_projection_point(w, seed: int, stream, hidden: int = 4096, rope_base: float = 500000.0):
    """The suffix QKV projection with rotary embedding, fused with the KV append
    (cw_qkv_rope_append), on the measured batch's suffix rows: an 8B-shaped
    layer (hidden 4096, 32 Q / 8 KV heads of 128, rope base 500000) with
    seeded random bf16 hidden states and weights. Algorithmic FLOPs are
    2 T hidden (Hq + 2 Hkv) D; bytes are x, W and the bf16 outputs once.
    hipBLASLt's time for the bare product x W^T is given for context."""
    import torch
    from paper_2606_19667_amd import batch as B
    from paper_2606_19667_amd import cw, inputs
    s = B.schedule(w)
    hq, hkv, D = w.num_q_heads, w.num_kv_heads, w.head_dim
    T = int(s.cu_suffix[-1])
    nf = (hq + 2 * hkv) * D
    meta = cw.BatchMeta(s.block_table, s.cu_suffix, s.prefix_len, hq, hkv, D)
    x = inputs.normal_bf16((seed, 101), (T, hidden), "cuda")
    wt = inputs.scaled_normal_bf16((seed, 102), (nf, hidden), hidden ** -0.5, "cuda")
    kc = torch.zeros((s.num_blocks, hkv, 16, D), dtype=torch.bfloat16, device="cuda")
    vc = torch.zeros((s.num_blocks, hkv, 16, D), dtype=torch.bfloat16, device="cuda")
    n_pos = int((s.prefix_len + np.diff(s.cu_suffix)).max())
    rope = torch.from_numpy(cw.rope_table(n_pos, D, rope_base)).cuda()
    q = torch.empty((T, hq, D), dtype=torch.bfloat16, device="cuda")
    fn = lambda: cw.qkv_rope_append(meta, x, wt, rope, kc, vc, q_out=q, stream=stream)
    for _ in range(5):
        fn()
    t = percentiles_us(timed_calls(fn, stream, 30))
    fl = 2.0 * T * hidden * nf
    by = 2 * (T * hidden + nf * hidden + T * nf)
    sec = t["median"] * 1e-6
    gemm = lambda: x @ wt.t()
    for _ in range(5):
        gemm()
    tg = percentiles_us(timed_calls(gemm, stream, 30))
    return {"kernel": "qkv_rope_append_kernel<128>", "tokens": T, "hidden": hidden, "features": nf,
            "us": t, "GFLOP": round(fl / 1e9, 2), "algorithmic_MB": round(by / 1e6, 1),
            "achieved_TFLOPs": round(fl / sec / 1e12, 1), "frac_bf16_peak": round(fl / sec / 1e12 / PEAK_BF16_TFLOPS, 4),
            "bound": "mfma", "gemm_only_hipblaslt_us": tg,
            "gemm_only_hipblaslt_TFLOPs": round(fl / (tg["median"] * 1e-6) / 1e12, 1)}


def cpu_model() -> str:
    """The host CPU's model name (first processor entry of /proc/cpuinfo)."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, sched, budget_s: float = 12.0):
    """The fp64 oracle on the host cores over whole requests of the batch, until
    about `budget_s` seconds have been spent (at least one request)."""
    from threadpoolctl import threadpool_info, threadpool_limits

    from oracle import attention as OA
    from paper_2606_19667_amd.workload import logical_kv, suffix_q

    cores = len(os.sched_getaffinity(0))
    flops = tokens = n = 0
    elapsed = 0.0
    with threadpool_limits(limits=cores):
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
        for r in range(w.batch):
            P = int(sched.prefix_len[r])
            k, v = logical_kv(w, w.prompts[r])
            q = suffix_q(w, w.prompts[r], P)
            t0 = time.perf_counter()
            OA.suffix_prefill_attention(q, k, v, P, w.scale)
            elapsed += time.perf_counter() - t0
            S = q.shape[0]
            flops += attention_flops([P], [S], w.num_q_heads, w.head_dim)
            tokens += S
            n += 1
            if elapsed >= budget_s:
                break
    return {"value": round(flops / elapsed / 1e12, 6), "unit": "TFLOP/s", "cores": int(threads),
            "kind": "oracle", "sample": f"{n} of {w.batch} requests (all heads and rows), fp64 NumPy",
            "cpu_model": cpu_model(),
            "seconds": round(elapsed, 3), "suffix_tokens_per_s": round(tokens / elapsed, 1)}


def copy_calibration(mbytes: int, reps: int = 5) -> None:
    """A plain device copy of `mbytes` MiB, `reps` times: the reference kernel
    whose FETCH_SIZE / WRITE_SIZE readings scale the attention kernel's."""
    import torch
    n = mbytes * (1 << 20) // 2
    a = torch.ones(n, dtype=torch.bfloat16, device="cuda")
    b = torch.empty_like(a)
    for _ in range(reps):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_MiB": mbytes, "reps": reps}), flush=True)


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="llama8b-trace-b16")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-diagnostic", action="store_true",
                    help="skip the question-only diagnostic point (keeps profiler passes to one workload)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MiB",
                    help="only run a plain device copy of this size (counter calibration)")
    args = ap.parse_args()
    if args.steps < 1 or args.warmup < 0:
        print("bench.py needs --steps >= 1 and --warmup >= 0", file=sys.stderr)
        return 2
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on one GPU only: this build has no multi-GPU path "
              "(requests, KV heads or prefix blocks would be sharded across GPUs; "
              "see the design notes).", file=sys.stderr)
        return 2

    import torch

    from paper_2606_19667_amd import batch as B
    from paper_2606_19667_amd import cw

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return 0
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] setting up {args.workload}", file=sys.stderr, flush=True)

    w = make_workload(args.workload, args.seed)
    stride = B.bt_stride_for(w)
    # Pool state after the warm-up queries were served: every step starts from it.
    snapshot = cw.Pool(w.num_blocks(), w.free_order())
    for p in w.warmup:
        bt0, pl0, cu0 = cw.schedule_batch(snapshot, [p.tokens(w.seed)], stride, w.block_size)
        cw.release_batch(snapshot, bt0, pl0, cu0, w.block_size)
    batch_tokens = [p.tokens(w.seed) for p in w.prompts]
    if w.prefix_lens is None:
        probe = snapshot.clone()
        sched = B.Scheduled(*cw.schedule_batch(probe, batch_tokens, stride, w.block_size), w.num_blocks())
        probe.close()
    else:
        sched = B.schedule(w)
    db = B.materialize(w, device=dev, keep_host=[], sched=sched,
                       gen_device="cuda" if w.num_q_heads * sum(p.length for p in w.prompts) > 2e7 else "cpu")
    hq, hkv, D = w.num_q_heads, w.num_kv_heads, w.head_dim
    S = np.diff(sched.cu_suffix)
    P = sched.prefix_len
    flops = attention_flops(P, S, hq, D)
    total_s = int(S.sum())

    stream = torch.cuda.current_stream()
    out = torch.empty_like(db.q)
    trace_mode = w.prefix_lens is None
    # Two runners alternate. A step's schedule goes up on a copy stream while
    # the previous step's kernels run: the upload of runner r waits until the
    # kernels of r's last step are done with its device buffer (ev_done), the
    # kernels wait for the upload (ev_up), and the host reuses r's pinned
    # buffer only once that upload has completed.
    copy_stream = torch.cuda.Stream(device=dev)

    def make_runners(fused: bool):
        rs = []
        for _ in range(2):
            rn = cw.BatchRunner([p.tokens(w.seed) for p in w.prompts], stride, hq, hkv, D, w.block_size,
                                device=dev, fused=fused)
            rn.bind(db.q, db.k_new, db.v_new, db.k_cache, db.v_cache, out, w.scale, stream=stream)
            rn.ev_up = None
            rn.ev_done = None
            rs.append(rn)
        return rs

    def step(runners, i: int, ev=None):
        rn = runners[i % 2]
        if rn.ev_up is not None:
            rn.ev_up.synchronize()
        pool = None
        if trace_mode:
            pool = snapshot.clone()
            rn.schedule(pool)
        else:
            rn.set_schedule(sched.block_table, sched.prefix_len, sched.cu_suffix)
        with torch.cuda.stream(copy_stream):
            if rn.ev_done is not None:
                copy_stream.wait_event(rn.ev_done)
            rn.upload()
            rn.ev_up = torch.cuda.Event()
            rn.ev_up.record(copy_stream)
        stream.wait_event(rn.ev_up)
        if rn.fused:
            if ev is not None:
                ev[0].record(stream)
            rn.append_attention()
            if ev is not None:
                ev[1].record(stream)
        elif ev is None:
            rn.kv_append()
            rn.attention()
        else:
            ev[0].record(stream)
            rn.kv_append()
            ev[1].record(stream)
            rn.attention()
            ev[2].record(stream)
        rn.ev_done = torch.cuda.Event()
        rn.ev_done.record(stream)
        if pool is not None:
            rn.release(pool)
            pool.close()

    def timed_steps(runners, warmup: int, settle_s: float):
        """Settle and warm-up steps, then args.steps timed steps (wall clock),
        then args.steps steps with HIP events around their kernels."""
        step(runners, 0)
        torch.cuda.synchronize()
        if runners[0].total_rows != total_s or not np.array_equal(runners[0].plen_host, P):
            raise RuntimeError("the scheduled batch differs from the prepared one")
        n_settle = 0
        t_settle = time.perf_counter()
        while time.perf_counter() - t_settle < settle_s:
            step(runners, n_settle)
            n_settle += 1
        for i in range(warmup):
            step(runners, i)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(args.steps):
            step(runners, i)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
        for i in range(args.steps):
            step(runners, args.steps + i, evs[i])
        torch.cuda.synchronize()
        return n_settle, ms, evs

    # The step: the fused append + attention call (cw_suffix_prefill_append_attn).
    # Settle: the card's clocks take tens of milliseconds of sustained load to
    # reach their steady state (the attention kernel runs ~20 % slower in the
    # first few milliseconds), so untimed steps run for at least SETTLE_S
    # seconds before the warm-up steps, whatever --warmup is.
    print(f"[bench] timing {args.steps} fused steps", file=sys.stderr, flush=True)
    fused_runners = make_runners(True)
    settle, ms_per_step, evs = timed_steps(fused_runners, args.warmup, SETTLE_S)
    fused_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    # The same steps with the two separate calls (cw_kv_append, then
    # cw_suffix_prefill_attn), for the per-kernel breakdown.
    print(f"[bench] timing {args.steps} steps of the separate calls", file=sys.stderr, flush=True)
    runners = make_runners(False)
    _, seq_ms_per_step, evs = timed_steps(runners, args.warmup, SETTLE_S)
    app_ms = sum(e[0].elapsed_time(e[1]) for e in evs) / args.steps
    attn_ms = sum(e[1].elapsed_time(e[2]) for e in evs) / args.steps

    rn = runners[(2 * args.steps - 1) % 2]
    print("[bench] per-call, cold-cache and host timings", file=sys.stderr, flush=True)
    # Per-call durations (hot caches) and with a 512 MB scratch buffer written
    # between calls, which evicts the K/V from L2 and the 256 MB MALL.
    hot = percentiles_us(timed_calls(rn.attention, stream, 50))
    fused_hot = percentiles_us(timed_calls(fused_runners[(2 * args.steps - 1) % 2].append_attention, stream, 50))
    scratch = torch.empty(256 << 20, dtype=torch.bfloat16, device=dev)
    cold = percentiles_us(timed_calls(rn.attention, stream, 20, between=lambda: scratch.fill_(1.0)))
    del scratch
    host = host_timing(w, snapshot, stride) if trace_mode else None

    achieved = flops / (fused_ms * 1e-3) / 1e12
    mfma_flops = executed_mfma_flops(sched.cu_suffix, P, hq, hkv, D)
    res = {
        "metric": "suffix-prefill attention TFLOP/s (whole step: schedule + KV append + attention)",
        "value": round(flops / (ms_per_step * 1e-3) / 1e12, 3),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_steps": settle,
        "ms_per_step": round(ms_per_step, 5),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.batch, "num_q_heads": hq, "num_kv_heads": hkv,
                   "head_dim": D, "block_size": w.block_size, "suffix_tokens": total_s,
                   "prefix_tokens": int(P.sum()), "prompt_tokens": int(P.sum()) + total_s,
                   "prefix_len": [int(x) for x in P]},
        "suffix_tokens_per_s": round(total_s / (ms_per_step * 1e-3), 1),
        "pct_bf16_peak_step": round(100 * flops / (ms_per_step * 1e-3) / 1e12 / PEAK_BF16_TFLOPS, 2),
        "step": "cw_suffix_prefill_append_attn (append and attention in one launch)",
        "append_attention_us": round(fused_ms * 1e3, 2),
        "separate_calls": {"ms_per_step": round(seq_ms_per_step, 5), "attention_us": round(attn_ms * 1e3, 2),
                           "kv_append_us": round(app_ms * 1e3, 2),
                           "kv_append_GBps": round(append_bytes(S, hkv, D) / (app_ms * 1e-3) / 1e9, 1),
                           "attention_TFLOPs": round(flops / (attn_ms * 1e-3) / 1e12, 3)},
        "attention_GFLOP": round(flops / 1e9, 3),
        "attention_mfma_GFLOP": round(mfma_flops / 1e9, 3),
        "mfma_waste_factor": round(mfma_flops / flops, 4),
        "roofline": {"bound": "mfma", "achieved": round(achieved, 3), "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": counted_traffic(args.workload),
                     "kernel": "suffix_prefill_attn_kernel<128, false, true>",
                     "algorithmic_bytes": int(attention_bytes(P, S, hq, hkv, D)) + append_bytes(S, hkv, D) // 2},
        "attention_call_us": hot,
        "append_attention_call_us": fused_hot,
        "attention_cold_us": cold,
    }
    if host is not None:
        res["host"] = host
    del db, runners, fused_runners, out
    torch.cuda.empty_cache()
    if args.workload == "llama8b-trace-b16" and not args.no_diagnostic:
        print("[bench] question-only diagnostic point", file=sys.stderr, flush=True)
        res["diagnostic_question_only"] = question_only_point(args.seed, stream)
        torch.cuda.empty_cache()
    if args.workload == "llama8b-trace-b16" and not args.no_diagnostic:
        print("[bench] other configurations (attention only)", file=sys.stderr, flush=True)
        res["configs"] = config_points(args.seed, stream)
    if args.workload == "llama8b-trace-b16" and not args.no_diagnostic:
        print("[bench] suffix QKV projection + rotary embedding + append", file=sys.stderr, flush=True)
        res["qkv_projection"] = qkv_projection_point(w, args.seed, stream)
        torch.cuda.empty_cache()
    if not args.no_diagnostic:
        print("[bench] sustained bf16 MFMA rate (measurement aid)", file=sys.stderr, flush=True)
        mp = mfma_peak_point(args.seed, stream)
        mp["attention_frac_of_normal_bf16"] = round(achieved / mp["normal_bf16"]["TFLOPs"], 4)
        res["mfma_peak_measured"] = mp
    if args.workload == "llama8b-trace-b16" and not args.no_diagnostic:
        print("[bench] ordering strategies and tight-pool replay (host)", file=sys.stderr, flush=True)
        res["ordering"] = ordering_point(args.seed)
    if not args.no_cpu_baseline:
        print("[bench] cpu baseline (fp64 oracle)", file=sys.stderr, flush=True)
        res["cpu_baseline"] = cpu_baseline(w, sched)
    print(json.dumps(res), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
