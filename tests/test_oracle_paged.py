"""Pins for the paged-cache oracle (not gpu).

Pools are built by scattering a padded cache into randomly permuted pool pages
(``workloads.to_pages``, which shares no code with the oracle's reads); the
paged oracle must then reproduce the padded oracle, itself pinned in
``test_oracle_attention.py`` / ``test_oracle_rope.py`` /
``test_oracle_select.py``.  Plausible slips in the table lookup, planted in the
oracle, must fail those comparisons.
"""
import numpy as np
import pytest

import oracle
import oracle.paged as OP
import workloads as W


def _inputs(P, seed=0, ctx=(70, 33, 100)):
    vi = W.random_verify_inputs(3, 4, 4, 2, 16, list(ctx), "f32", seed=seed)
    rows = vi.ctx_len.astype(np.int64) + 4
    table, n_pages = W.page_table(rows, P, seed=seed)
    kp = W.to_pages(vi.k.astype(np.float64), table, n_pages, P)
    vp = W.to_pages(vi.v.astype(np.float64), table, n_pages, P)
    return vi, table, n_pages, kp, vp


def _paged_matches_padded(vi, table, kp, vp, P):
    out, lse, mass = OP.verify_attn_paged(vi.q, kp, vp, table, vi.ctx_len, vi.scale, P)
    ro, rl, rm = oracle.verify_attn(vi.q, vi.k, vi.v, vi.ctx_len, vi.scale)
    n = rm.shape[1]
    return (np.allclose(out, ro, rtol=0, atol=1e-12) and np.allclose(lse, rl, rtol=0, atol=1e-12)
            and np.allclose(mass[:, :n], rm, rtol=0, atol=1e-12) and not mass[:, n:].any())


@pytest.mark.parametrize("P", [32, 64])
def test_verify_paged_equals_padded(P):
    vi, table, _, kp, vp = _inputs(P)
    assert (table[:, 1:] != table[:, :-1] + 1).any()      # pages really are scattered
    assert _paged_matches_padded(vi, table, kp, vp, P)


def test_verify_paged_pool_permutation_invariant():
    """Relabelling pool pages (pool and table together) changes nothing."""
    P = 32
    vi, table, n_pages, kp, vp = _inputs(P, seed=3)
    perm = np.random.default_rng(5).permutation(n_pages)
    t2 = np.where(table >= 0, perm[np.maximum(table, 0)], -1).astype(np.int32)
    kp2, vp2 = np.zeros_like(kp), np.zeros_like(vp)
    kp2[perm], vp2[perm] = kp, vp
    a = OP.verify_attn_paged(vi.q, kp, vp, table, vi.ctx_len, vi.scale, P)
    b = OP.verify_attn_paged(vi.q, kp2, vp2, t2, vi.ctx_len, vi.scale, P)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


def test_lookup_slips_fail(monkeypatch):
    P = 32
    vi, table, _, kp, vp = _inputs(P, seed=1)
    good = OP._page_of
    slips = {
        "offset_off_by_one": lambda t, b, i, P: (good(t, b, i, P)[0], (i + 1) % P),
        "batch_ignored": lambda t, b, i, P: (int(t[0, i // P]), i % P),
        "page_size_off": lambda t, b, i, P: (int(t[b, i // (P // 2) % t.shape[1]]), i % P),
        "logical_page_as_pool": lambda t, b, i, P: (i // P, i % P),
    }
    for name, slip in slips.items():
        monkeypatch.setattr(OP, "_page_of", slip)
        try:
            ok = _paged_matches_padded(vi, table, kp, vp, P)
        except IndexError:
            ok = False
        assert not ok, name
    monkeypatch.setattr(OP, "_page_of", good)
    assert _paged_matches_padded(vi, table, kp, vp, P)


def test_rope_append_paged_equals_padded():
    P = 32
    B, T, Hq, Hkv, D = 3, 4, 4, 2, 16
    rng = np.random.default_rng(2)
    ctx = np.array([70, 33, 100], np.int32)
    n_cap = int(ctx.max()) + T
    q = rng.standard_normal((B, T, Hq, D))
    kn = rng.standard_normal((B, T, Hkv, D))
    vn = rng.standard_normal((B, T, Hkv, D))
    kc = rng.standard_normal((B, Hkv, n_cap, D))
    vc = rng.standard_normal((B, Hkv, n_cap, D))
    pos = (ctx[:, None] + np.arange(T)[None]).astype(np.int32)
    table, n_pages = W.page_table(ctx + T, P, seed=4)
    qo, kr, vr = oracle.rope.rope_append(q, kn, vn, pos, ctx, kc, vc, 1e6)
    qp, kpr, vpr = OP.rope_append_paged(q, kn, vn, pos, ctx, W.to_pages(kc, table, n_pages, P),
                                        W.to_pages(vc, table, n_pages, P), table, P, 1e6)
    assert np.array_equal(qo, qp)
    assert np.array_equal(W.to_pages(kr, table, n_pages, P), kpr)
    assert np.array_equal(W.to_pages(vr, table, n_pages, P), vpr)


def test_gather_paged_equals_padded_stacked():
    P = 64
    L, B, Hkv, D = 2, 3, 2, 8
    rng = np.random.default_rng(6)
    rows = np.array([150, 64, 200])
    n_cap = int(rows.max())
    kc = rng.integers(0, 65535, size=(L, B, Hkv, n_cap, D)).astype(np.uint16)
    vc = rng.integers(0, 65535, size=(L, B, Hkv, n_cap, D)).astype(np.uint16)
    table, n_pages = W.page_table(rows, P, seed=7)
    K = np.array([20, 0, 33], np.int32)
    idx = np.zeros((B, 40), np.int32)
    for b in range(B):
        idx[b, :K[b]] = np.sort(rng.choice(rows[b] - 10, size=K[b], replace=False))
    tb = rows.astype(np.int32) - 10
    tl = np.full(B, 10, np.int32)
    kd, vd = OP.gather_kv_paged(W.to_pages(kc, table, n_pages, P), W.to_pages(vc, table, n_pages, P),
                                table, P, idx, K, tb, tl, 50)
    for l in range(L):
        rk, rv = oracle.gather_kv(kc[l], vc[l], idx, K, tb, tl, 50)
        assert np.array_equal(kd[l], rk) and np.array_equal(vd[l], rv)
