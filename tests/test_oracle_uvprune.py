"""Pins for the UV-Prune oracle (not gpu): Eq. (similarity) and
Eq. (average_similarity), checked against hand-computed fixtures,
scikit-learn's cosine_similarity, and identities that hold for the exact
definition (scale invariance, linearity of the text sum, telescoping of the
layer sum, cancellation of a per-position bias)."""
import numpy as np
import pytest
from sklearn.metrics.pairwise import cosine_similarity

import oracle
from golden_io import similarity_fixture


def test_golden_cosines():
    fx = similarity_fixture()
    for a, b, e in fx["cos"]:
        assert oracle.cos_similarity(a, b) == pytest.approx(e, abs=1e-15)


def test_golden_criterion_and_score():
    fx = similarity_fixture()
    V = fx["crit_V"].reshape(1, 2, 2)
    X = fx["crit_X"].reshape(1, 2, 2)
    c = oracle.criterion_cossim(V, X, [2], [2])
    np.testing.assert_allclose(c[0], fx["crit_c"], rtol=1e-15)
    hv = np.stack([fx["score_V0"].reshape(1, 2, 2), fx["score_V1"].reshape(1, 2, 2)])
    ht = np.stack([fx["score_X0"].reshape(1, 1, 2), fx["score_X1"].reshape(1, 1, 2)])
    s = oracle.uvprune_score_cossim(hv, ht, [2], [1])
    np.testing.assert_allclose(s[0], fx["score"], rtol=1e-15, atol=1e-16)


def test_against_sklearn():
    rng = np.random.default_rng(0)
    hv = rng.standard_normal((2, 30, 17))
    ht = rng.standard_normal((2, 9, 17))
    hv[0, 4] = 0.0        # zero-norm visual row
    ht[1, 2] = 0.0        # zero-norm text row
    c = oracle.criterion_cossim(hv, ht, [30, 25], [9, 7])
    for b, (mb, nb) in enumerate([(30, 9), (25, 7)]):
        ref = cosine_similarity(hv[b, :mb], ht[b, :nb]).sum(axis=1)
        np.testing.assert_allclose(c[b, :mb], ref, rtol=1e-12, atol=1e-13)
        assert np.all(c[b, mb:] == 0.0)


def test_identical_tokens_give_n():
    rng = np.random.default_rng(1)
    x = rng.standard_normal(12)
    hv = np.tile(x, (1, 5, 1))
    ht = np.tile(2.5 * x, (1, 7, 1))
    c = oracle.criterion_cossim(hv, ht, [5], [7])
    np.testing.assert_allclose(c[0], 7.0, rtol=1e-14)


def test_scale_invariance_and_linearity():
    rng = np.random.default_rng(2)
    hv = rng.standard_normal((1, 20, 11))
    ht = rng.standard_normal((1, 6, 11))
    c = oracle.criterion_cossim(hv, ht, [20], [6])
    scales_v = rng.uniform(0.1, 10, size=(1, 20, 1))
    scales_t = rng.uniform(0.1, 10, size=(1, 6, 1))
    c2 = oracle.criterion_cossim(hv * scales_v, ht * scales_t, [20], [6])
    np.testing.assert_allclose(c, c2, rtol=1e-12, atol=1e-14)
    u = (ht[0] / np.linalg.norm(ht[0], axis=1, keepdims=True)).sum(axis=0)
    lin = (hv[0] / np.linalg.norm(hv[0], axis=1, keepdims=True)) @ u
    np.testing.assert_allclose(c[0], lin, rtol=1e-12, atol=1e-14)


def test_telescoping_and_L1():
    rng = np.random.default_rng(3)
    L = 4
    hv = rng.standard_normal((L + 1, 2, 15, 8))
    ht = rng.standard_normal((L + 1, 2, 5, 8))
    m, n = [15, 12], [5, 4]
    s = oracle.uvprune_score_cossim(hv, ht, m, n)
    cL = oracle.criterion_cossim(hv[L], ht[L], m, n)
    c0 = oracle.criterion_cossim(hv[0], ht[0], m, n)
    np.testing.assert_allclose(s, cL - c0, rtol=1e-11, atol=1e-13)
    s1 = oracle.uvprune_score_cossim(hv[:2], ht[:2], m, n)
    c1 = oracle.criterion_cossim(hv[1], ht[1], m, n)
    np.testing.assert_allclose(s1, c1 - c0, rtol=1e-12, atol=1e-13)


def test_mass_variation_properties():
    rng = np.random.default_rng(4)
    crit = rng.random((6, 3, 40))
    m = [40, 33, 1]
    s = oracle.uvprune_score_mass(crit, m)
    for b, mb in enumerate(m):
        np.testing.assert_allclose(s[b, :mb], crit[5, b, :mb] - crit[0, b, :mb], rtol=1e-12, atol=1e-14)
        assert np.all(s[b, mb:] == 0.0)
    bias = rng.standard_normal((1, 3, 40)) * 100.0
    np.testing.assert_allclose(oracle.uvprune_score_mass(crit + bias, m), s, rtol=1e-9, atol=1e-11)
    # explicit differences of a hand-made stack
    hand = np.array([[[1.0, 2.0]], [[4.0, 1.0]], [[2.0, 7.0]]])
    np.testing.assert_allclose(oracle.uvprune_score_mass(hand, [2])[0], [1.0, 5.0])


# ---- the prefill epilogue (residual add + criterion of the stored result) --
def test_round_to_storage_matches_torch_bf16():
    """The oracle's bf16 rounding (round to nearest even, through fp32) equals
    torch's conversion, a library routine, on random values, exact ties and
    values near the fp32 limits."""
    import torch
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.standard_normal(20000) * 10.0 ** rng.integers(-30, 30, 20000),
                        (np.arange(-300, 300) + 0.5) * 2.0 ** -7,      # exact bf16 ties
                        [3.0e38, -3.0e38, 1e-38, -1e-40, 0.0, -0.0]])
    mine = oracle.uvprune.round_to_storage(x, "bf16")
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    assert np.array_equal(mine, ref)
    assert np.array_equal(oracle.uvprune.round_to_storage(x, "f32"), x.astype(np.float32).astype(np.float64))


def test_prefill_epilogue_pins():
    rng = np.random.default_rng(4)
    B, m_cap, n_cap, D = 2, 9, 5, 16
    m, n = np.array([9, 4]), np.array([5, 2])
    bf = lambda a: oracle.uvprune.round_to_storage(a, "bf16")
    vp, vd = bf(rng.standard_normal((B, m_cap, D))), bf(rng.standard_normal((B, m_cap, D)))
    tp, td = bf(rng.standard_normal((B, n_cap, D))), bf(rng.standard_normal((B, n_cap, D)))
    # a zero delta leaves the rows and gives the plain criterion of them
    hv, ht, c = oracle.prefill_epilogue(vp, 0 * vd, tp, 0 * td, m, n, "bf16")
    assert np.array_equal(hv, vp) and np.array_equal(ht, tp)
    assert np.array_equal(c, oracle.criterion_cossim(vp, tp, m, n))
    # small integers add exactly: the rounding is then the identity
    ip = rng.integers(-50, 50, (B, m_cap, D)).astype(np.float64)
    idl = rng.integers(-50, 50, (B, m_cap, D)).astype(np.float64)
    hv, _, _ = oracle.prefill_epilogue(ip, idl, tp, td, m, n, "bf16")
    assert np.array_equal(hv[0], ip[0] + idl[0]) and np.array_equal(hv[1, :4], ip[1, :4] + idl[1, :4])
    # rows past m / n are not written
    hv, ht, c = oracle.prefill_epilogue(vp, vd, tp, td, m, n, "bf16")
    assert np.array_equal(hv[1, 4:], vp[1, 4:]) and np.array_equal(ht[1, 2:], tp[1, 2:])
    assert not c[1, 4:].any()
    # the criterion is that of the rounded sums, not of the exact ones
    exact = oracle.criterion_cossim(vp + vd, tp + td, m, n)
    assert np.array_equal(c, oracle.criterion_cossim(bf(vp + vd), ht, m, n))
    assert not np.array_equal(c, exact)
