"""Pins for the speculative accept/reject oracle (not gpu).

Checked against what the mathematics of speculative sampling fixes:
hand-derived fixtures; greedy acceptance reproducing the target's argmax
chain (the lossless property, Sec. 2.2); the per-position acceptance
probability sum_x min(p, q) and the emitted-token law p, both by seeded
Monte Carlo; and forced accept/reject cases.
"""
import math

import numpy as np
import pytest

import oracle
from golden_io import accept_fixture


def _logits(p):
    return np.log(np.asarray(p, dtype=np.float64)).astype(np.float32)


def test_golden_cases():
    fx = accept_fixture()
    dl = _logits(fx["q1"])[None, None, :]
    tl = np.stack([_logits(fx["p1"]), _logits(fx["p2"])])[None]
    toks = np.array([[int(fx["x"][0])]], dtype=np.int32)
    for ua, us, na, nt in fx["cases"]:
        n, y, tie = oracle.spec_accept(dl, tl, toks, np.array([[ua]]), np.array([us]), 1.0)
        assert (int(n[0]), int(y[0])) == (na, nt), (ua, us)
        assert tie[0] == 0


def test_greedy_reproduces_target_argmax_chain():
    rng = np.random.default_rng(0)
    B, g, V = 6, 5, 50
    tl = rng.standard_normal((B, g + 1, V)).astype(np.float32)
    dl = rng.standard_normal((B, g, V)).astype(np.float32)
    am = tl.argmax(axis=-1)
    toks = np.zeros((B, g), dtype=np.int32)
    for b in range(B):
        j = b % (g + 1)                 # first j drafts agree with the target
        toks[b] = am[b, :g]
        if j < g:
            toks[b, j] = (am[b, j] + 1) % V
    n, y, _ = oracle.spec_accept(dl, tl, toks, rng.random((B, g)), rng.random(B), 0.0)
    for b in range(B):
        j = b % (g + 1)
        assert n[b] == j
        assert y[b] == am[b, j]
        emitted = list(toks[b, :n[b]]) + [int(y[b])]
        assert emitted == list(am[b, :n[b] + 1])


def test_greedy_tie_lowest_index():
    tl = np.zeros((1, 2, 4), dtype=np.float32)
    tl[0, 0, [1, 3]] = 2.0
    tl[0, 1, [2, 3]] = 5.0
    n, y, _ = oracle.spec_accept(np.zeros((1, 1, 4), np.float32), tl,
                                 np.array([[1]], np.int32), np.zeros((1, 1)), np.zeros(1), 0.0)
    assert (n[0], y[0]) == (1, 2)


def _mc(p_logits, q_logits, trials, seed):
    rng = np.random.default_rng(seed)
    V = p_logits.shape[-1]
    q = oracle.softmax_t(q_logits, 1.0)
    toks = rng.choice(V, size=trials, p=q).astype(np.int32)
    dl = np.broadcast_to(q_logits, (trials, 1, V))
    tl = np.broadcast_to(np.stack([p_logits, p_logits]), (trials, 2, V))
    return oracle.spec_accept(dl, tl, toks[:, None], rng.random((trials, 1)), rng.random(trials), 1.0), toks


def test_acceptance_rate_and_output_law():
    V = 6
    p_logits = np.array([1.2, -0.3, 0.5, 2.0, -1.0, 0.1], np.float32)
    q_logits = np.array([0.2, 0.9, 0.4, 0.6, 0.5, -0.7], np.float32)
    trials = 60000
    (n, y, _), toks = _mc(p_logits, q_logits, trials, 1)
    p = oracle.softmax_t(p_logits, 1.0)
    q = oracle.softmax_t(q_logits, 1.0)
    alpha = np.minimum(p, q).sum()
    sigma = math.sqrt(alpha * (1 - alpha) / trials)
    assert abs(n.mean() - alpha) < 4.5 * sigma
    first = np.where(n == 1, toks, y)          # first emitted token
    counts = np.bincount(first, minlength=V)
    chi2 = ((counts - trials * p) ** 2 / (trials * p)).sum()
    assert chi2 < 25.7                          # chi-square(5) at p = 1e-4
    bonus = y[n == 1]                           # bonus token law is p as well
    cb = np.bincount(bonus, minlength=V)
    chi2b = ((cb - len(bonus) * p) ** 2 / (len(bonus) * p)).sum()
    assert chi2b < 25.7


def test_forced_cases():
    V = 5
    rng = np.random.default_rng(4)
    z = rng.standard_normal((1, 3, V)).astype(np.float32)
    toks = np.array([[1, 2, 3]], np.int32)
    n, _, _ = oracle.spec_accept(z[:, :3], np.concatenate([z, z[:, :1]], axis=1), toks,
                                 np.full((1, 3), 1 - 2.0 ** -53), np.array([0.5]), 1.0)
    assert n[0] == 3                        # p = q: every draft accepted
    tl = np.concatenate([z, z[:, :1]], axis=1).copy()
    tl[0, 1, 2] = -np.inf                   # p(x) = 0 at position 2
    n, y, _ = oracle.spec_accept(z[:, :3], tl, toks, np.zeros((1, 3)), np.array([0.5]), 1.0)
    assert n[0] == 1 and y[0] != 2
    tl = np.concatenate([z, z[:, :1]], axis=1).copy()
    tl[0, 0, 1] -= 3.0                      # p(x) < q(x) at position 1
    n, _, _ = oracle.spec_accept(z[:, :3], tl, toks, np.full((1, 3), 1 - 2.0 ** -53),
                                 np.array([0.5]), 1.0)
    assert n[0] == 0


def test_near_tie_flag():
    p = np.log(np.array([0.5, 0.5])).astype(np.float32)
    q = np.log(np.array([0.25, 0.75])).astype(np.float32)
    pv = oracle.softmax_t(p, 1.0)
    qv = oracle.softmax_t(q, 1.0)
    u = pv[1] / qv[1]                        # u * q(x) == p(x) up to rounding
    _, _, tie = oracle.spec_accept(q[None, None], np.stack([p, p])[None],
                                   np.array([[1]], np.int32), np.array([[u]]), np.array([0.3]), 1.0)
    assert tie[0] == 1


# ---- temperature (Sec. 2.2 rule with p and q at temperature tau) ----------
def _tempered_fixture():
    fx = accept_fixture("spec_accept_temperature.txt")
    tau = float(fx["tau"][0])
    dl = (tau * np.log(fx["q1"]))[None, None, :].astype(np.float32)
    tl = np.stack([tau * np.log(fx["p1"]), tau * np.log(fx["p2"])])[None].astype(np.float32)
    toks = np.array([[int(fx["x"][0])]], dtype=np.int32)
    return fx, tau, dl, tl, toks


def _fixture_mismatches(fn, fx, tau, dl, tl, toks):
    bad = 0
    for ua, us, na, nt in fx["cases"]:
        n, y, _ = fn(dl, tl, toks, np.array([[ua]]), np.array([us]), tau)
        bad += (int(n[0]), int(y[0])) != (na, nt)
    return bad


def test_golden_cases_at_temperature():
    fx, tau, dl, tl, toks = _tempered_fixture()
    for ua, us, na, nt in fx["cases"]:
        n, y, tie = oracle.spec_accept(dl, tl, toks, np.array([[ua]]), np.array([us]), tau)
        assert (int(n[0]), int(y[0])) == (na, nt), (ua, us)
        assert tie[0] == 0


def test_temperature_slips_fail_the_fixture(monkeypatch):
    """Each plausible temperature slip, planted in the oracle, fails at least
    one hand-derived case: the fixture pins the scaling, not just the rule."""
    import oracle.accept as A
    fx, tau, dl, tl, toks = _tempered_fixture()
    assert _fixture_mismatches(oracle.spec_accept, fx, tau, dl, tl, toks) == 0
    good = A.softmax_t

    def times_tau(z, t):
        return good(np.asarray(z, np.float64) * t * t, t)    # softmax(z * tau)

    def untempered(z, t):
        return good(np.asarray(z, np.float64) * t, t)        # softmax(z)

    for slip in (times_tau, untempered):
        monkeypatch.setattr(A, "softmax_t", slip)
        assert _fixture_mismatches(A.spec_accept, fx, tau, dl, tl, toks) > 0, slip.__name__
    monkeypatch.setattr(A, "softmax_t", good)
    # only one of p and q tempered: the other's logits effectively unscaled
    q_only = lambda d, t_, *r: A.spec_accept(d, (t_ * tau).astype(np.float32), *r)
    p_only = lambda d, t_, *r: A.spec_accept((d * tau).astype(np.float32), t_, *r)
    for slip in (q_only, p_only):
        assert _fixture_mismatches(slip, fx, tau, dl, tl, toks) > 0


def test_acceptance_rate_and_output_law_at_temperature():
    """tau = 0.7: per-position acceptance probability sum_x min(p_tau, q_tau)
    and the emitted-token law p_tau, with p_tau and q_tau from torch.softmax in
    float64 (a library routine independent of the oracle's softmax)."""
    import torch
    tau = float(np.float32(0.7))   # the oracle takes the temperature as float32
    V = 6
    p_logits = np.array([1.2, -0.3, 0.5, 2.0, -1.0, 0.1], np.float32)
    q_logits = np.array([0.2, 0.9, 0.4, 0.6, 0.5, -0.7], np.float32)
    p = torch.softmax(torch.from_numpy(p_logits.astype(np.float64)) / tau, 0).numpy()
    q = torch.softmax(torch.from_numpy(q_logits.astype(np.float64)) / tau, 0).numpy()
    trials = 60000
    rng = np.random.default_rng(7)
    toks = rng.choice(V, size=trials, p=q).astype(np.int32)
    dl = np.broadcast_to(q_logits, (trials, 1, V))
    tl = np.broadcast_to(np.stack([p_logits, p_logits]), (trials, 2, V))
    n, y, _ = oracle.spec_accept(dl, tl, toks[:, None], rng.random((trials, 1)), rng.random(trials), tau)
    alpha = np.minimum(p, q).sum()
    sigma = math.sqrt(alpha * (1 - alpha) / trials)
    assert abs(n.mean() - alpha) < 4.5 * sigma
    # the untempered rate differs by far more than the band: the test sees tau
    p1, q1 = oracle.softmax_t(p_logits, 1.0), oracle.softmax_t(q_logits, 1.0)
    assert abs(np.minimum(p1, q1).sum() - alpha) > 10 * sigma
    first = np.where(n == 1, toks, y)
    counts = np.bincount(first, minlength=V)
    chi2 = ((counts - trials * p) ** 2 / (trials * p)).sum()
    assert chi2 < 25.7                          # chi-square(5) at p = 1e-4
