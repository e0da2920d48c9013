"""Parity of pvlm_window_size and pvlm_speedup (C library) with the oracle.

These two calls are host arithmetic (no device pointer, no stream), so the
comparison runs without a GPU.  Windows must match exactly; the speedup
model's times and speedups within 1e-9 relative (the library sums Lemma 1's
series where the oracle takes its closed form).
"""
import math

import numpy as np
import pytest

import paper_2603_19610_amd as P
from golden_io import window_fixture
from oracle import window as W

REL = 1e-9


def _oracle_model(c, tau, g):
    t = {
        "t_sd_ideal": W.t_sd_ideal(c, g),
        "t_psd_ideal": W.t_psd_ideal(c, g),
        "t_sd": W.t_sd_practical(c, tau, g),
        "t_psd": W.t_psd_practical(c, tau, g),
        "t_psd_rollback": W.t_psd_rollback(c, tau, g),
    }
    out = dict(t)
    for k, v in t.items():
        out["v" + k[1:]] = W.speedup(c, v)
    out["expected_accepted"] = W.expected_accepted(tau, g)
    out["expected_total"] = W.expected_total(tau, g)
    return out


def _close(a, b):
    if math.isinf(b):
        return math.isinf(a)
    return a == pytest.approx(b, rel=REL, abs=1e-300)


def _cases():
    rng = np.random.default_rng(2603_19610)
    cases = [(c, tau, g) for c in (0.4, 1.0, 1.36, 5.0, 5.36, 9.01, 33.3)
             for tau in (0.0, 0.05, 0.5, 0.9, 0.999, 1.0) for g in (1, 2, 5, 9, 17, 64)]
    for _ in range(300):
        cases.append((float(rng.uniform(0.2, 40.0)), float(rng.uniform(0.0, 1.0)),
                      int(rng.integers(1, 200))))
    return cases


def test_speedup_model_matches_oracle():
    for c, tau, g in _cases():
        got = P.speedup(c, tau, g)
        want = _oracle_model(c, tau, g)
        bad = [k for k in want if not _close(got[k], want[k])]
        assert not bad, (c, tau, g, {k: (got[k], want[k]) for k in bad})


def test_window_size_matches_oracle_on_printed_tables():
    fx = window_fixture()
    for pair, alpha, t_p, t_q, _ in fx["ratio"] + fx["gamma"]:
        for mode in ("down", "up", "nearest"):
            g, c = P.window_size(t_p, t_q, mode)
            assert g == W.window_size(t_p, t_q, mode), (pair, alpha, mode)
            assert c == W.speed_ratio(t_p, t_q)
        for tau in (0.3, 0.6, 0.8, 0.9, 0.95, 1.0):
            assert P.window_size(t_p, t_q, "best", tau)[0] == \
                W.window_size(t_p, t_q, "best", tau=tau), (pair, alpha, tau)
    for t_p, t_q, g in fx["example"]:
        assert P.window_size(t_p, t_q, "nearest")[0] == int(g)


def test_window_size_matches_oracle_random_and_edges():
    rng = np.random.default_rng(7)
    cases = [(0.3, 0.1), (10, 4), (1, 4), (1000, 1), (7, 7), (5, 1), (6, 1)]
    cases += [(float(rng.uniform(1, 500)), float(rng.uniform(1, 100))) for _ in range(300)]
    for t_p, t_q in cases:
        for gmax in (1, 3, 16, 64):
            for mode in ("down", "up", "nearest"):
                assert P.window_size(t_p, t_q, mode, gamma_max=gmax)[0] == \
                    W.window_size(t_p, t_q, mode, gamma_max=gmax), (t_p, t_q, mode, gmax)
            for tau in (0.01, 0.4, 0.77, 0.93, 1.0):
                assert P.window_size(t_p, t_q, "best", tau, gmax)[0] == \
                    W.window_size(t_p, t_q, "best", tau=tau, gamma_max=gmax), \
                    (t_p, t_q, tau, gmax)


@pytest.mark.parametrize("args", [
    (0.0, 0.5, 4), (-1.0, 0.5, 4), (math.inf, 0.5, 4), (math.nan, 0.5, 4),
    (2.0, -0.1, 4), (2.0, 1.5, 4), (2.0, math.nan, 4), (2.0, 0.5, 0), (2.0, 0.5, (1 << 20) + 1),
])
def test_speedup_rejects_bad_arguments(args):
    with pytest.raises(P.PvlmError) as e:
        P.speedup(*args)
    assert e.value.status == 2


@pytest.mark.parametrize("args", [
    (0.0, 1.0, "down", 0.0, 64), (1.0, 0.0, "down", 0.0, 64), (math.inf, 1.0, "up", 0.0, 64),
    (1.0, math.nan, "up", 0.0, 64), (1.0, 1.0, "down", 0.0, 0), (1.0, 1.0, "best", 0.0, 64),
    (1.0, 1.0, "best", 1.5, 64), (1e300, 1e-300, "down", 0.0, 64),
])
def test_window_size_rejects_bad_arguments(args):
    with pytest.raises(P.PvlmError) as e:
        P.window_size(*args)
    assert e.value.status == 2


def test_window_size_null_and_unknown_mode():
    import ctypes
    L = P.lib()
    assert L.pvlm_window_size(4.0, 1.0, 0, 0.0, 64, None, None) == 1
    g = ctypes.c_int(0)
    assert L.pvlm_window_size(4.0, 1.0, 9, 0.0, 64, ctypes.byref(g), None) == 2
    assert L.pvlm_speedup(4.0, 0.5, 4, None) == 1
