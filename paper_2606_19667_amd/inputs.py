"""Seeded synthetic inputs shared by the library's tests, bench and oracle checks.

This module draws random numbers and token IDs from integer keys and nothing
else: it holds none of the attention, hashing or block-table arithmetic. Every
array it returns is a pure function of its key, so two calls with the same key
give identical bits on any machine.

* Values are N(0, 1) drawn in float32 and rounded to bfloat16 (round to
  nearest even, torch's conversion).
* Token IDs are uniform in [0, vocab).
* A key is a tuple of non-negative ints; numpy's SeedSequence turns it into the
  seed of an independent stream.
"""
from __future__ import annotations

import numpy as np
import torch

VOCAB = 1 << 17


def _seed64(key) -> int:
    state = np.random.SeedSequence([int(x) for x in key]).generate_state(2, dtype=np.uint32)
    return int(state[0]) | (int(state[1]) << 32)


def normal_bf16(key, shape, device="cpu") -> torch.Tensor:
    """bfloat16 tensor of N(0, 1) draws for `key` (drawn on `device`)."""
    g = torch.Generator(device=device)
    g.manual_seed(_seed64(key) & ((1 << 63) - 1))
    x = torch.randn(tuple(shape), generator=g, dtype=torch.float32, device=device)
    return x.to(torch.bfloat16)


def scaled_normal_bf16(key, shape, std: float, device="cpu") -> torch.Tensor:
    """bfloat16 tensor of N(0, std^2) draws for `key`: std times an N(0, 1) draw
    in float32, then rounded (weights of a linear layer use std = fan_in^-1/2)."""
    g = torch.Generator(device=device)
    g.manual_seed(_seed64(key) & ((1 << 63) - 1))
    x = torch.randn(tuple(shape), generator=g, dtype=torch.float32, device=device)
    return (x * float(std)).to(torch.bfloat16)


def token_ids(key, n: int, vocab: int = VOCAB) -> np.ndarray:
    """int32 token IDs for `key`."""
    rng = np.random.default_rng(np.random.SeedSequence([int(x) for x in key]))
    return rng.integers(0, vocab, size=int(n), dtype=np.int64).astype(np.int32)


def rng(key) -> np.random.Generator:
    """numpy Generator for structural draws (placements, trace choices)."""
    return np.random.default_rng(np.random.SeedSequence([int(x) for x in key]))


def permutation(key, n: int) -> np.ndarray:
    """A seeded permutation of range(n) (int32)."""
    return rng(key).permutation(int(n)).astype(np.int32)
