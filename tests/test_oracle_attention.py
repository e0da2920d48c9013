"""Pins for the verify-attention oracle (not gpu).

The oracle is checked against things other than itself: hand-computed
fixtures, a brute-force scalar implementation, PyTorch's
scaled_dot_product_attention and softmax in float64, and closed forms
(mass conservation, uniform keys, a single visible key).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from golden_io import verify_cases


def _rand(seed, B, T, Hq, Hkv, D, ctx):
    rng = np.random.default_rng(seed)
    n_cap = max(ctx) + T + 3
    q = rng.standard_normal((B, T, Hq, D))
    k = rng.standard_normal((B, Hkv, n_cap, D))
    v = rng.standard_normal((B, Hkv, n_cap, D))
    return q, k, v, np.array(ctx, dtype=np.int64)


@pytest.mark.parametrize("case", verify_cases(), ids=lambda c: c["name"])
def test_golden_fixture(case):
    D, Hq, Hkv, T, ctx = (int(case[k][0]) for k in ("D", "Hq", "Hkv", "T", "ctx_len"))
    n = ctx + T
    q = case["q"].reshape(1, T, Hq, D)
    k = case["k"].reshape(1, Hkv, n, D)
    v = case["v"].reshape(1, Hkv, n, D)
    out, lse, mass = oracle.verify_attn(q, k, v, [ctx], float(case["scale"][0]))
    np.testing.assert_allclose(out.reshape(-1), case["out"], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(lse.reshape(-1), case["lse"], rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(mass.reshape(-1), case["mass"], rtol=1e-14, atol=1e-15)


def _brute(q, k, v, ctx, scale):
    B, T, Hq, D = q.shape
    Hkv = k.shape[1]
    out = np.zeros_like(q)
    mass = np.zeros((B, k.shape[2]))
    lse = np.zeros((B, Hq, T))
    for b in range(B):
        for h in range(Hq):
            g = h // (Hq // Hkv)
            for t in range(T):
                rows = range(int(ctx[b]) + t + 1)
                s = [scale * sum(q[b, t, h, d] * k[b, g, i, d] for d in range(D)) for i in rows]
                z = sum(math.exp(x) for x in s)
                for i in rows:
                    p = math.exp(s[i]) / z
                    mass[b, i] += p
                    for d in range(D):
                        out[b, t, h, d] += p * v[b, g, i, d]
                lse[b, h, t] = math.log(z)
    return out, lse, mass


def test_brute_force_tiny():
    q, k, v, ctx = _rand(1, 2, 3, 4, 2, 5, [4, 6])
    o1, l1, m1 = oracle.verify_attn(q, k, v, ctx, 0.37)
    o2, l2, m2 = _brute(q, k, v, ctx, 0.37)
    np.testing.assert_allclose(o1, o2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(l1, l2, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(m1, m2, rtol=1e-12, atol=1e-13)


@pytest.mark.parametrize("shape", [(1, 5, 4, 1, 16, [40]), (2, 9, 8, 2, 32, [33, 57]),
                                   (3, 1, 6, 3, 8, [0, 5, 11])])
def test_against_torch_sdpa(shape):
    B, T, Hq, Hkv, D, ctx = shape
    q, k, v, ctx = _rand(7, B, T, Hq, Hkv, D, ctx)
    scale = 1.0 / math.sqrt(D)
    out, lse, mass = oracle.verify_attn(q, k, v, ctx, scale)
    n_cap = k.shape[2]
    G = Hq // Hkv
    for b in range(B):
        qt = torch.from_numpy(q[b]).permute(1, 0, 2)                      # [Hq][T][D]
        kt = torch.from_numpy(k[b]).repeat_interleave(G, dim=0)          # [Hq][n][D]
        vt = torch.from_numpy(v[b]).repeat_interleave(G, dim=0)
        t_idx = torch.arange(T)[:, None]
        i_idx = torch.arange(n_cap)[None, :]
        allowed = i_idx <= (int(ctx[b]) + t_idx)                          # [T][n]
        ref = torch.nn.functional.scaled_dot_product_attention(
            qt, kt, vt, attn_mask=allowed, scale=scale)
        np.testing.assert_allclose(out[b], ref.permute(1, 0, 2).numpy(), rtol=1e-11, atol=1e-12)
        scores = torch.einsum("htd,hnd->htn", qt, kt) * scale
        scores = scores.masked_fill(~allowed, float("-inf"))
        np.testing.assert_allclose(lse[b], torch.logsumexp(scores, dim=-1).numpy(),
                                   rtol=1e-12, atol=1e-12)
        P = torch.softmax(scores, dim=-1)
        np.testing.assert_allclose(mass[b], P.sum(dim=(0, 1)).numpy(), rtol=1e-11, atol=1e-13)


def test_mass_conservation_and_masking():
    q, k, v, ctx = _rand(3, 2, 6, 8, 2, 16, [20, 31])
    _, _, mass = oracle.verify_attn(q, k, v, ctx, 0.25)
    Hq, T = 8, 6
    for b in range(2):
        assert mass[b].sum() == pytest.approx(Hq * T, rel=1e-13)
        assert np.all(mass[b, int(ctx[b]) + T:] == 0.0)
        assert np.all(mass[b, :int(ctx[b]) + T] > 0.0)


def test_uniform_keys_closed_form():
    B, T, Hq, Hkv, D = 1, 4, 6, 2, 8
    ctx = 10
    rng = np.random.default_rng(5)
    q = rng.standard_normal((B, T, Hq, D))
    k = np.tile(rng.standard_normal(D), (B, Hkv, ctx + T, 1))
    v = rng.standard_normal((B, Hkv, ctx + T, D))
    out, lse, mass = oracle.verify_attn(q, k, v, [ctx], 0.5)
    for h in range(Hq):
        g = h // (Hq // Hkv)
        for t in range(T):
            n = ctx + t + 1
            np.testing.assert_allclose(out[0, t, h], v[0, g, :n].mean(axis=0), rtol=1e-12, atol=1e-13)
            s = 0.5 * float(q[0, t, h] @ k[0, g, 0])
            assert lse[0, h, t] == pytest.approx(s + math.log(n), rel=1e-13)
    expect = np.array([sum(Hq / (ctx + t + 1) for t in range(T) if i <= ctx + t)
                       for i in range(ctx + T)])
    np.testing.assert_allclose(mass[0], expect, rtol=1e-13)


def test_single_visible_key_is_plain_decode():
    q, k, v, _ = _rand(11, 1, 1, 4, 1, 8, [0])
    out, lse, mass = oracle.verify_attn(q, k, v, [0], 0.3)
    for h in range(4):
        np.testing.assert_allclose(out[0, 0, h], v[0, 0, 0], rtol=1e-15)
        assert lse[0, h, 0] == pytest.approx(0.3 * float(q[0, 0, h] @ k[0, 0, 0]))
    assert mass[0, 0] == pytest.approx(4.0)


def test_rows_sampler_matches_full():
    q, k, v, ctx = _rand(13, 2, 3, 4, 2, 8, [9, 14])
    out, lse, mass = oracle.verify_attn(q, k, v, ctx, 0.4)
    res = oracle.verify_attn_rows(q, k, v, ctx, 0.4, [(1, 3, 2), (0, 0, 0)])
    np.testing.assert_allclose(res[(1, 3, 2)][0], out[1, 2, 3], rtol=1e-14)
    assert res[(0, 0, 0)][1] == pytest.approx(lse[0, 0, 0], rel=1e-15)
