"""Seeded generator checks (not gpu): determinism, shapes, keep counts and
the bf16 rounding against torch's own float32 -> bfloat16 conversion."""
import numpy as np
import torch

import workloads as W


def test_keep_counts_and_shapes():
    w = W.WORKLOADS
    assert int(w["tiny"].keep_count([768])[0]) == 192
    assert int(w["llava7b"].keep_count([6272])[0]) == 627
    assert int(w["llava72b"].keep_count([12544])[0]) == 1254
    assert int(w["long"].keep_count([131072])[0]) == 3932
    q = w["qwen32b"]
    lens = q.lengths()
    assert lens.shape == (4,) and lens.min() >= 16384 and lens.max() <= 33280
    assert np.array_equal(q.keep_count(q.m_per_seq()), (lens - 512) // 20)
    assert w["llava72b"].T == 9 and w["llava72b"].group == 8


def test_determinism_and_layout():
    w = W.WORKLOADS["tiny"]
    a = W.make_verify_inputs(w, layer=1)
    b = W.make_verify_inputs(w, layer=1)
    assert np.array_equal(a.k, b.k) and np.array_equal(a.q, b.q)
    assert a.q.shape == (1, 5, 4, 64) and a.k.shape == (1, 1, 1029, 64)
    assert a.k.dtype == np.float32 and int(a.ctx_len[0]) == 1024
    z = W.make_verify_inputs(w, layer=0)
    assert not np.array_equal(z.k, a.k)          # salient boost only on layer 1
    assert np.array_equal(z.v, a.v)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = np.concatenate([rng.standard_normal(10000) * 10.0 ** rng.integers(-30, 30, 10000),
                        [0.0, -0.0, np.inf, -np.inf, 1.00390625, 1.01171875]]).astype(np.float32)
    mine = W.f32_to_bf16_bits(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, ref)
    back = W.bf16_bits_to_f64(mine)
    assert np.array_equal(back, torch.from_numpy(x).to(torch.bfloat16).double().numpy())


def test_rope_is_a_rotation():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 64))
    y = W.rope_f64(x, np.arange(7) * 1000, 1.0e6)
    np.testing.assert_allclose(np.linalg.norm(y, axis=1), np.linalg.norm(x, axis=1), rtol=1e-13)
    np.testing.assert_allclose(y[0], x[0])
    # relative-position property: <R(a) x, R(b) y> depends on b - a only
    u, v = rng.standard_normal(64), rng.standard_normal(64)
    d1 = W.rope_f64(u, 5, 1e4) @ W.rope_f64(v, 9, 1e4)
    d2 = W.rope_f64(u, 105, 1e4) @ W.rope_f64(v, 109, 1e4)
    assert abs(d1 - d2) < 1e-10


def test_accept_inputs():
    w = W.WORKLOADS["tiny"]
    a = W.make_accept_inputs(w)
    assert a.draft_logits.shape == (1, 4, 1024) and a.target_logits.shape == (1, 5, 1024)
    assert a.draft_tokens.dtype == np.int32 and a.u_accept.dtype == np.float64
    g = W.make_accept_inputs(w, temperature=0.0)
    assert np.array_equal(g.draft_tokens[0], g.draft_logits[0].argmax(axis=-1))
