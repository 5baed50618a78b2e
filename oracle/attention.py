"""fp64 reference for causal prefill of a suffix over a cached prefix.

TEST INFRASTRUCTURE ONLY (see the package docstring).

Definition followed (paper Sec. 1 and 2.1; Sec. 3.3 after Eq. 1): prefix
caching reuses the KV states of the leading P tokens of a prompt, so only the S
suffix tokens are prefilled, and the result must equal what a from-scratch
prefill of all P + S tokens gives for those rows: prefix reuse changes cost,
not what the model sees. The paper does not write out the attention itself; it
is standard scaled-dot-product causal attention over the serving engine's KV
blocks. The readings taken here:

* suffix row i sits at absolute position P + i and sees keys 0 .. P + i
  (bottom-right alignment of the causal mask);
* grouped-query attention with contiguous groups: query head h reads KV head
  h // (Hq / Hkv);
* softmax scale is an explicit argument (1/sqrt(D) in every workload);
* inputs are the logical sequences (never a device cache); every value is
  upcast exactly to float64 and the result is returned in float64.
"""
from __future__ import annotations

import math

import numpy as np


def _as_f64(x) -> np.ndarray:
    """Exact upcast of a float array (numpy or torch, any float dtype) to float64."""
    if hasattr(x, "detach"):  # torch tensor; bf16 has no numpy dtype
        x = x.detach().to("cpu").double().numpy()
    return np.asarray(x, dtype=np.float64)


def _attend_rows(q_rows: np.ndarray, k: np.ndarray, v: np.ndarray, row_pos: np.ndarray,
                 scale: float) -> np.ndarray:
    """Rows of attention: query rows q_rows [R, Hq, D] at absolute positions
    row_pos [R] over keys/values k, v [L, Hkv, D]; row n sees keys 0 .. row_pos[n]."""
    R, Hq, D = q_rows.shape
    L, Hkv, _ = k.shape
    G = Hq // Hkv
    out = np.zeros((R, Hq, D), dtype=np.float64)
    visible = np.arange(L)[None, :] <= row_pos[:, None]           # [R, L]
    for g in range(Hkv):
        qg = q_rows[:, g * G:(g + 1) * G, :]                         # [R, G, D]
        scores = scale * (qg @ k[:, g, :].T)                         # [R, G, L]
        scores = np.where(visible[:, None, :], scores, -np.inf)
        m = scores.max(axis=2, keepdims=True)
        w = np.exp(scores - m)                                       # exp(-inf) = 0
        out[:, g * G:(g + 1) * G, :] = (w @ v[:, g, :]) / w.sum(axis=2, keepdims=True)
    return out


def _check_shapes(q, k, v, prefix_len):
    S, Hq, D = q.shape
    L, Hkv, Dk = k.shape
    if Dk != D or v.shape != k.shape:
        raise ValueError("k/v shape mismatch")
    if L != prefix_len + S:
        raise ValueError(f"logical length {L} != prefix {prefix_len} + suffix {S}")
    if Hq % Hkv:
        raise ValueError("Hq must be a multiple of Hkv")


def suffix_prefill_attention(q, k, v, prefix_len: int, scale: float,
                             row_chunk: int = 256) -> np.ndarray:
    """Attention output of the S suffix rows of one request.

    q: [S, Hq, D] suffix queries; k, v: [L, Hkv, D] logical keys/values of the
    whole prompt (L = prefix_len + S, prefix first). Returns [S, Hq, D] float64.

    For each query head h (KV head g = h // G) and suffix row i:
        s_j = scale * <q[i, h], k[j, g]>           for j = 0 .. prefix_len + i
        O[i, h] = sum_j exp(s_j - max s) v[j, g] / sum_j exp(s_j - max s)
    Rows are processed in chunks of `row_chunk` only to bound memory; each row's
    arithmetic is independent of the chunking.
    """
    q = _as_f64(q)
    k = _as_f64(k)
    v = _as_f64(v)
    _check_shapes(q, k, v, prefix_len)
    S = q.shape[0]
    out = np.zeros(q.shape, dtype=np.float64)
    for r0 in range(0, S, row_chunk):
        r1 = min(S, r0 + row_chunk)
        out[r0:r1] = _attend_rows(q[r0:r1], k, v, prefix_len + np.arange(r0, r1), scale)
    return out


def suffix_prefill_attention_loops(q, k, v, prefix_len: int, scale: float) -> np.ndarray:
    """The same definition written as plain Python loops (tiny inputs only)."""
    q = _as_f64(q)
    k = _as_f64(k)
    v = _as_f64(v)
    S, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    out = np.zeros((S, Hq, D), dtype=np.float64)
    for i in range(S):
        pos = prefix_len + i
        for h in range(Hq):
            g = h // G
            s = []
            for j in range(pos + 1):
                acc = 0.0
                for d in range(D):
                    acc += float(q[i, h, d]) * float(k[j, g, d])
                s.append(scale * acc)
            m = max(s)
            w = [math.exp(x - m) for x in s]
            tot = sum(w)
            for d in range(D):
                acc = 0.0
                for j in range(pos + 1):
                    acc += w[j] * float(v[j, g, d])
                out[i, h, d] = acc / tot
    return out


def suffix_prefill_rows(q, k, v, prefix_len: int, scale: float, rows,
                        row_chunk: int = 256) -> np.ndarray:
    """Output of selected suffix rows only: [len(rows), Hq, D] float64.

    Each row depends only on its own query and keys 0 .. prefix_len + row, so a
    sampled row is computed exactly as in the full call. q holds all S rows.
    """
    q = _as_f64(q)
    k = _as_f64(k)
    v = _as_f64(v)
    rows = np.asarray(rows, dtype=np.int64)
    _check_shapes(q, k, v, prefix_len)
    q_sel = q[rows]
    out = np.zeros((len(rows),) + q.shape[1:], dtype=np.float64)
    for r0 in range(0, len(rows), row_chunk):
        r1 = min(len(rows), r0 + row_chunk)
        out[r0:r1] = _attend_rows(q_sel[r0:r1], k, v, prefix_len + rows[r0:r1], scale)
    return out


def attention_flops(prefix_lens, suffix_lens, num_q_heads: int, head_dim: int) -> int:
    """Algorithmic FLOPs of the visible (query, key) pairs: QK^T and PV
    multiply-adds, 4 * D * Hq * sum_r (S_r * P_r + S_r (S_r + 1) / 2)."""
    pairs = 0
    for p, s in zip(prefix_lens, suffix_lens):
        pairs += s * p + s * (s + 1) // 2
    return 4 * head_dim * num_q_heads * pairs


# ---------------------------------------------------------------------------
# Attention over a subset of the keys, and the log-sum-exp merge of such parts.
#
# Softmax over a union of disjoint key sets factors through per-set sums: with
# Z_A = sum_{j in A} exp(s_j), softmax over A u B weights the set-A output
# O_A = sum_{j in A} exp(s_j) v_j / Z_A by Z_A / (Z_A + Z_B). The parts are
# therefore kept as (O_A, log Z_A); the merge is the definition of the softmax
# written through those sums. The library reports log Z in base 2
# (log2 Z = ln Z / ln 2), and so do these functions.
# ---------------------------------------------------------------------------
def suffix_prefill_partial(q, k, v, prefix_len: int, scale: float, key_lo: int, key_hi: int):
    """Attention of the suffix rows over the keys j in [key_lo, key_hi) that
    each row may see (j <= prefix_len + i).

    Returns (o [S, Hq, D], lse2 [S, Hq]) in float64: o is normalised over the
    part's visible keys and lse2 = log2(sum_j exp(s_j)) over them; a row that
    sees none of the part's keys gets o = 0 and lse2 = -inf.
    """
    q = _as_f64(q)
    k = _as_f64(k)
    v = _as_f64(v)
    _check_shapes(q, k, v, prefix_len)
    S, Hq, D = q.shape
    L, Hkv, _ = k.shape
    G = Hq // Hkv
    o = np.zeros((S, Hq, D), dtype=np.float64)
    lse2 = np.full((S, Hq), -np.inf, dtype=np.float64)
    j = np.arange(L)
    for i in range(S):
        keys = j[(j >= key_lo) & (j < key_hi) & (j <= prefix_len + i)]
        if keys.size == 0:
            continue
        for h in range(Hq):
            g = h // G
            s = scale * (k[keys, g, :] @ q[i, h, :])
            m = s.max()
            w = np.exp(s - m)
            o[i, h] = (w @ v[keys, g, :]) / w.sum()
            lse2[i, h] = (m + math.log(w.sum())) / math.log(2.0)
    return o, lse2


def lse_merge(parts_o, parts_lse2) -> np.ndarray:
    """Combine parts computed over disjoint key sets.

    parts_o [n, rows, D], parts_lse2 [n, rows] (base 2, -inf for an empty
    part) -> [rows, D]: sum_p 2^(lse_p) o_p / sum_p 2^(lse_p), evaluated
    relative to the largest lse_p; a row with every part empty is zero.
    """
    o = _as_f64(parts_o)
    lse = _as_f64(parts_lse2)
    m = lse.max(axis=0)                                              # [rows]
    finite = np.isfinite(m)
    w = np.where(np.isfinite(lse), np.exp2(lse - np.where(finite, m, 0.0)[None, :]), 0.0)   # [n, rows]
    tot = w.sum(axis=0)
    out = np.einsum("pr,prd->rd", w, o)
    return np.where(tot[:, None] > 0, out / np.where(tot > 0, tot, 1.0)[:, None], 0.0)
