"""Host-side helpers of bench.py on the CPU: algorithmic FLOPs, the executed
MFMA FLOPs of the attention kernel's tile plan, and the --gpus contract."""
import os
import subprocess
import sys

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_executed_mfma_flops_by_hand():
    # 4 query heads on one KV head (G = 4): a tile holds 256 / 4 = 64 positions.
    # Request 0: P = 64, S = 32 -> one tile, keys 0 .. 95 -> 2 steps of 64 keys.
    # Request 1: P = 0, S = 100 -> tiles at rows 0 and 64: keys 0 .. 63 (1 step)
    # and 0 .. 99 (2 steps). Each step is 256 rows x 64 keys x D x 4 FLOPs.
    cu = np.array([0, 32, 132], dtype=np.int32)
    plen = np.array([64, 0], dtype=np.int32)
    D = 64
    got = bench.executed_mfma_flops(cu, plen, 4, 1, D)
    assert got == (2 + 1 + 2) * 256 * 64 * D * 4
    # the same with 2 KV heads doubles every tile
    assert bench.executed_mfma_flops(cu, plen, 8, 2, D) == 2 * got


def test_executed_exceeds_algorithmic():
    cu = np.array([0, 576], dtype=np.int32)
    plen = np.array([832], dtype=np.int32)
    alg = bench.attention_flops(plen, np.diff(cu), 32, 128)
    ex = bench.executed_mfma_flops(cu, plen, 32, 8, 128)
    assert ex >= alg
    assert ex / alg < 1.2


def test_more_than_one_gpu_is_refused():
    p = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert p.returncode != 0
    assert "one GPU" in (p.stdout + p.stderr) or "1 GPU" in (p.stdout + p.stderr)
