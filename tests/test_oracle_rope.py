"""Pins for the RoPE / M-RoPE append oracle (not gpu).

Checked against what the definition fixes, each written independently of the
oracle's complex product: the explicit 2x2 rotation matrix of every pair;
position 0 is the identity; every pair keeps its norm; the score of a rotated
query and key depends only on the position difference (the relative property
RoPE is built for); M-RoPE with equal temporal, height and width positions is
1-D RoPE, and with one section covering every pair it follows that axis only;
the append writes exactly rows ctx_len .. ctx_len + T - 1.
"""
import math

import numpy as np
import pytest

from oracle import rope as R

BASE = 1.0e6


def _matrix_rope(x, p, base):
    """Pair by pair with the rotation matrix [[cos, -sin], [sin, cos]]."""
    D = x.shape[-1]
    h = D // 2
    y = np.empty(D)
    for i in range(h):
        a = p[i] * base ** (-2.0 * i / D)
        c, s = math.cos(a), math.sin(a)
        y[i] = c * x[i] - s * x[i + h]
        y[i + h] = s * x[i] + c * x[i + h]
    return y


def test_matches_rotation_matrices():
    rng = np.random.default_rng(1)
    for D in (8, 64, 128):
        x = rng.standard_normal(D)
        for sections in (None, (D // 8, D // 8 * 1, D // 2 - D // 4)):
            pos = np.array([13.0, 7.0, 99.0]) if sections else np.array(4321.0)
            pp = R.pair_positions(pos, D, sections)
            np.testing.assert_allclose(R.rotate(x, pp, BASE), _matrix_rope(x, pp, BASE),
                                       rtol=0, atol=1e-12)


def test_identity_and_norms():
    rng = np.random.default_rng(2)
    x = rng.standard_normal((5, 128))
    np.testing.assert_allclose(R.rotate(x, np.zeros((5, 64)), BASE), x, atol=0)
    y = R.rotate(x, rng.integers(0, 200000, (5, 64)).astype(float), BASE)
    np.testing.assert_allclose(y[:, :64] ** 2 + y[:, 64:] ** 2, x[:, :64] ** 2 + x[:, 64:] ** 2,
                               rtol=1e-12)


def test_relative_position_property():
    rng = np.random.default_rng(3)
    q, k = rng.standard_normal(64), rng.standard_normal(64)

    def score(pq, pk):
        return R.rotate(q, R.pair_positions(np.array(float(pq)), 64), 1e4) @ \
            R.rotate(k, R.pair_positions(np.array(float(pk)), 64), 1e4)
    for d in (0, 1, 17, 500):
        vals = [score(p + d, p) for p in (0, 3, 1000, 12345)]
        np.testing.assert_allclose(vals, vals[0], rtol=1e-9)
    assert abs(score(5, 0) - score(0, 5)) > 1e-6   # not symmetric in general


def test_mrope_reduces_to_1d_and_follows_one_axis():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((3, 128))
    p = np.array([7.0, 300.0, 41000.0])
    one_d = R.rotate(x, R.pair_positions(p, 128), BASE)
    m = R.rotate(x, R.pair_positions(np.stack([p, p, p]), 128, (16, 24, 24)), BASE)
    np.testing.assert_allclose(m, one_d, atol=0)
    three = np.stack([p, p + 5, p + 9])
    for a, sec in enumerate(((64, 0, 0), (0, 64, 0), (0, 0, 64))):
        m = R.rotate(x, R.pair_positions(three, 128, sec), BASE)
        np.testing.assert_allclose(m, R.rotate(x, R.pair_positions(three[a], 128), BASE),
                                   atol=0)
    # the (16, 24, 24) split: pair 15 follows t, pair 16 h, pair 40 w
    pp = R.pair_positions(three, 128, (16, 24, 24))
    assert pp[0, 15] == 7 and pp[0, 16] == 12 and pp[0, 39] == 12 and pp[0, 40] == 16


def test_append_rows():
    rng = np.random.default_rng(5)
    B, T, Hq, Hkv, D, n_cap = 2, 3, 4, 2, 16, 12
    q = rng.standard_normal((B, T, Hq, D))
    kn, vn = rng.standard_normal((B, T, Hkv, D)), rng.standard_normal((B, T, Hkv, D))
    kc, vc = rng.standard_normal((B, Hkv, n_cap, D)), rng.standard_normal((B, Hkv, n_cap, D))
    ctx = np.array([0, 9])
    pos = np.array([[0, 1, 2], [20, 21, 22]])
    q2, kc2, vc2 = R.rope_append(q, kn, vn, pos, ctx, kc, vc, 1e4)
    for b in range(B):
        rows = set(range(ctx[b], ctx[b] + T))
        for r in range(n_cap):
            if r not in rows:
                assert np.array_equal(kc2[b, :, r], kc[b, :, r])
                assert np.array_equal(vc2[b, :, r], vc[b, :, r])
        for t in range(T):
            assert np.array_equal(vc2[b, :, ctx[b] + t], vn[b, t])
            for g in range(Hkv):
                np.testing.assert_allclose(kc2[b, g, ctx[b] + t],
                                           _matrix_rope(kn[b, t, g], [pos[b, t]] * 8, 1e4),
                                           atol=1e-12)
            for h in range(Hq):
                np.testing.assert_allclose(q2[b, t, h], _matrix_rope(q[b, t, h], [pos[b, t]] * 8,
                                                                     1e4), atol=1e-12)
    # position 0 rotates nothing
    assert np.allclose(kc2[0, :, 0], kn[0, 0])
