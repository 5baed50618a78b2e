"""fp64 reference for the suffix QKV projection with rotary position embedding.

TEST INFRASTRUCTURE ONLY (see the package docstring).

What it follows: a prefix hit removes the per-layer prefill work of the cached
tokens, and the work that remains for the suffix starts with projecting each
suffix token's hidden state to its query, key and value heads (paper Sec. 1
and Sec. 2.1: only the uncached suffix is prefilled; the measured models are
Qwen2.5 decoder-only transformers, Sec. 4). The paper does not write out the
layer; the readings taken here are the ones its model family uses:

* y = x W^T (+ b): x [T, hidden], W [(Hq + 2 Hkv) D, hidden] (the weight of a
  linear layer, one row per output feature), b an optional bias [(Hq + 2 Hkv) D];
  features [0, Hq D) are the query heads, then Hkv key heads, then Hkv value
  heads, each D wide;
* rotary embedding on queries and keys at the token's absolute position p, in
  the rotate-half form: for j < D/2, with theta_j = base^(-2j/D),
    out[j]       = u[j] cos(p theta_j) - u[j + D/2] sin(p theta_j)
    out[j + D/2] = u[j + D/2] cos(p theta_j) + u[j] sin(p theta_j);
  values are not rotated;
* suffix row i of request r sits at position P_r + i.

Everything is computed in float64 from exact upcasts of the inputs.
"""
from __future__ import annotations

import numpy as np


def _as_f64(x) -> np.ndarray:
    if hasattr(x, "detach"):
        x = x.detach().to("cpu").double().numpy()
    return np.asarray(x, dtype=np.float64)


def rope_angles(positions, head_dim: int, base: float) -> np.ndarray:
    """p * theta_j for every position p and j < D/2: [len(positions), D/2] fp64."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    theta = np.power(float(base), -2.0 * j / head_dim)
    return np.asarray(positions, dtype=np.float64)[:, None] * theta[None, :]


def rope(u, positions, base: float) -> np.ndarray:
    """Rotate-half rotary embedding of u [T, H, D] at positions [T]."""
    u = _as_f64(u)
    D = u.shape[-1]
    h = D // 2
    ang = rope_angles(positions, D, base)[:, None, :]
    c, s = np.cos(ang), np.sin(ang)
    a, b = u[..., :h], u[..., h:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def project(x, w, bias=None) -> np.ndarray:
    """y = x W^T (+ b) in float64."""
    y = _as_f64(x) @ _as_f64(w).T
    if bias is not None:
        y = y + _as_f64(bias)[None, :]
    return y


def qkv_rope(x, w, positions, num_q_heads: int, num_kv_heads: int, head_dim: int,
             base: float, bias=None):
    """(q [T, Hq, D], k [T, Hkv, D], v [T, Hkv, D]) in float64: the projection,
    split into heads, with the rotary embedding applied to q and k."""
    y = project(x, w, bias)
    T = y.shape[0]
    nq, nk = num_q_heads * head_dim, num_kv_heads * head_dim
    q = y[:, :nq].reshape(T, num_q_heads, head_dim)
    k = y[:, nq:nq + nk].reshape(T, num_kv_heads, head_dim)
    v = y[:, nq + nk:nq + 2 * nk].reshape(T, num_kv_heads, head_dim)
    return rope(q, positions, base), rope(k, positions, base), v


def suffix_positions(cu_suffix, prefix_len) -> np.ndarray:
    """Absolute position of every suffix row: P_r + i for row cu[r] + i."""
    out = []
    for r in range(len(prefix_len)):
        n = int(cu_suffix[r + 1]) - int(cu_suffix[r])
        out.append(int(prefix_len[r]) + np.arange(n))
    return np.concatenate(out).astype(np.int64) if out else np.zeros(0, np.int64)
