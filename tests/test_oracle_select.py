"""Pins for the Top-K and gather oracles (not gpu): hand-ranked fixtures,
numpy's stable argsort (which orders -0.0 equal to +0.0 and NaN last, as the
readings require), permutation equivariance and identity gathers."""
import numpy as np
import pytest

import oracle
import workloads
from golden_io import topk_fixture


def test_golden_ranking():
    for grp in topk_fixture():
        s = grp["scores"][None, :]
        for k, expect in grp["k"]:
            idx = oracle.topk_select(s, [s.shape[1]], [k], s.shape[1])
            assert list(idx[0, :k]) == expect
            assert np.all(idx[0, k:] == -1)


@pytest.mark.parametrize("kind", ["normal", "ties", "zeros", "special"])
def test_against_numpy_stable_argsort(kind):
    s = workloads.make_scores(3, 257, kind, seed=1)
    m = [257, 200, 31]
    k = [40, 200, 0]
    idx = oracle.topk_select(s, m, k, 210)
    for b in range(3):
        ref = np.sort(np.argsort(-s[b, :m[b]].astype(np.float64), kind="stable")[:k[b]])
        assert list(idx[b, :k[b]]) == list(ref)
        assert np.all(idx[b, k[b]:] == -1)


def test_permutation_equivariance():
    rng = np.random.default_rng(2)
    s = rng.standard_normal(100).astype(np.float32)      # distinct values
    perm = rng.permutation(100)
    a = oracle.topk_select(s[None], [100], [17], 17)[0]
    b = oracle.topk_select(s[perm][None], [100], [17], 17)[0]
    assert sorted(perm[b]) == list(a)


def test_k_equals_m_and_zero():
    s = workloads.make_scores(1, 50, "normal")
    assert list(oracle.topk_select(s, [50], [50], 50)[0]) == list(range(50))
    assert np.all(oracle.topk_select(s, [50], [0], 4)[0] == -1)


def test_gather_identity_and_tail():
    rng = np.random.default_rng(3)
    k = rng.integers(0, 65535, size=(2, 3, 20, 8), dtype=np.uint16)
    v = rng.integers(0, 65535, size=(2, 3, 20, 8), dtype=np.uint16)
    idx = np.tile(np.arange(20, dtype=np.int32), (2, 1))
    kd, vd = oracle.gather_kv(k, v, idx, [20, 20], [0, 0], [0, 0], 20)
    assert np.array_equal(kd, k) and np.array_equal(vd, v)
    idx = np.array([[1, 5, 7, -1], [0, 2, -1, -1]], dtype=np.int32)
    kd, vd = oracle.gather_kv(k, v, idx, [3, 2], [15, 10], [4, 2], 8)
    assert np.array_equal(kd[0, :, :3], k[0, :, [1, 5, 7]].transpose(1, 0, 2))
    assert np.array_equal(kd[0, :, 3:7], k[0, :, 15:19])
    assert np.array_equal(vd[1, :, 2:4], v[1, :, 10:12])
    assert np.all(kd[1, :, 4:] == 0)
