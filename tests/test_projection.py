"""Suffix QKV projection with rotary embedding (CPU part).

Pins the fp64 oracle (oracle.projection) to facts that do not come from
itself: hand-worked rotations for D = 2 and 4, the identity at position 0,
pairwise norm preservation, the relative-position property of the rotation,
composition of rotations, a complex-number formulation, basis-vector and
small-integer projections, and the head split. Then checks the library's
host-built cos/sin table against fp64 angles.
"""
import math

import numpy as np
import pytest

from oracle import projection as PR
from paper_2606_19667_amd import cw


def test_rope_identity_at_position_zero():
    u = np.random.default_rng(0).standard_normal((3, 2, 8))
    assert np.array_equal(PR.rope(u, [0, 0, 0], 10000.0), u)


def test_rope_hand_examples():
    for p in (1, 2, 7):
        out = PR.rope(np.array([[[1.0, 0.0]]]), [p], 500000.0)[0, 0]      # theta_0 = 1
        assert np.allclose(out, [math.cos(p), math.sin(p)], atol=1e-15)
        out = PR.rope(np.array([[[0.0, 1.0]]]), [p], 500000.0)[0, 0]
        assert np.allclose(out, [-math.sin(p), math.cos(p)], atol=1e-15)
    # D = 4, base 100: theta = (1, 0.1); pairs are (0, 2) and (1, 3)
    e0 = PR.rope(np.array([[[1.0, 0.0, 0.0, 0.0]]]), [2], 100.0)[0, 0]
    assert np.allclose(e0, [math.cos(2), 0, math.sin(2), 0], atol=1e-15)
    e1 = PR.rope(np.array([[[0.0, 1.0, 0.0, 0.0]]]), [2], 100.0)[0, 0]
    assert np.allclose(e1, [0, math.cos(0.2), 0, math.sin(0.2)], atol=1e-15)


def test_rope_preserves_pair_norms_and_matches_complex_rotation():
    rng = np.random.default_rng(1)
    u = rng.standard_normal((5, 3, 16))
    pos = np.array([0, 3, 100, 4095, 10367])
    out = PR.rope(u, pos, 500000.0)
    h = 8
    assert np.allclose(out[..., :h] ** 2 + out[..., h:] ** 2, u[..., :h] ** 2 + u[..., h:] ** 2, atol=1e-12)
    theta = 500000.0 ** (-2.0 * np.arange(h) / 16)
    z = (u[..., :h] + 1j * u[..., h:]) * np.exp(1j * pos[:, None, None] * theta[None, None, :])
    assert np.allclose(out[..., :h], z.real, atol=1e-12) and np.allclose(out[..., h:], z.imag, atol=1e-12)


def test_rope_scores_depend_on_relative_position_and_compose():
    rng = np.random.default_rng(2)
    q, k = rng.standard_normal((1, 1, 64)), rng.standard_normal((1, 1, 64))
    base = 10000.0
    dots = []
    for m, n in ((5, 2), (105, 102), (3000, 2997)):
        dots.append(float((PR.rope(q, [m], base) * PR.rope(k, [n], base)).sum()))
    assert np.allclose(dots, dots[0], atol=1e-10)
    assert np.allclose(PR.rope(PR.rope(q, [17], base), [25], base), PR.rope(q, [42], base), atol=1e-12)


def test_projection_basis_vectors_and_small_integers():
    rng = np.random.default_rng(3)
    w = rng.standard_normal((12, 6))
    b = rng.standard_normal(12)
    y = PR.project(np.eye(6), w, b)
    assert np.allclose(y, w.T + b[None, :], atol=0)
    x = np.array([[1.0, 2.0, -1.0]])
    w2 = np.array([[1.0, 0.0, 0.0], [2.0, 1.0, 1.0], [0.0, -3.0, 4.0]])
    assert PR.project(x, w2).tolist() == [[1.0, 3.0, -10.0]]     # hand-computed rows of w2 . x


def test_qkv_split_order_and_value_heads_unrotated():
    Hq, Hkv, D = 4, 2, 8
    N = (Hq + 2 * Hkv) * D
    x = np.random.default_rng(4).standard_normal((3, N))
    w = np.eye(N)                                        # y = x: features in order q | k | v
    pos = [0, 9, 30]
    q, k, v = PR.qkv_rope(x, w, pos, Hq, Hkv, D, 10000.0)
    assert np.allclose(q, PR.rope(x[:, :Hq * D].reshape(3, Hq, D), pos, 10000.0))
    assert np.allclose(k, PR.rope(x[:, Hq * D:(Hq + Hkv) * D].reshape(3, Hkv, D), pos, 10000.0))
    assert np.array_equal(v, x[:, (Hq + Hkv) * D:].reshape(3, Hkv, D))


def test_suffix_positions():
    assert PR.suffix_positions([0, 3, 3, 5], [16, 0, 32]).tolist() == [16, 17, 18, 32, 33]


@pytest.mark.parametrize("D,base", [(64, 10000.0), (128, 500000.0), (128, 1e6)])
def test_rope_table_matches_fp64_angles(D, base):
    n = 10400
    tab = cw.rope_table(n, D, base)
    assert tab.shape == (n, D // 2, 2) and tab.dtype == np.float32
    ang = PR.rope_angles(np.arange(n), D, base)
    ref = np.stack([np.cos(ang), np.sin(ang)], axis=-1)
    # one fp32 rounding of the fp64 values (a libm may differ in the last fp64 bit)
    assert np.abs(tab.astype(np.float64) - ref).max() <= 2.0 ** -24
