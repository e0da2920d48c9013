"""Pins for the window-size and speedup oracle (not gpu).

Checked against what the paper prints and what the mathematics fixes: the
supplement's table of exact speed ratios and the main text's integer windows
(tests/golden/window_size.txt); the worked example under Eq. (Prefill); Lemma
1's mean and the rollback proof's two-round token count by exhaustive
enumeration of acceptance vectors; the closed form the supplement gives for
the rollback speedup at gamma = c; and the special cases in which the
practical theorems reduce to the ideal ones.
"""
import itertools
import math

import pytest

from golden_io import window_fixture
from oracle import window as W

TAUS = (0.05, 0.3, 0.5, 0.83, 0.99, 1.0)


def test_printed_speed_ratios():
    fx = window_fixture()
    assert len(fx["ratio"]) == 15
    nearest = 0
    for pair, alpha, t_p, t_q, printed in fx["ratio"]:
        c = W.speed_ratio(t_p, t_q)
        # printed to one decimal: within one digit of the exact quotient
        lo, hi = math.floor(10 * c + 1e-9) / 10, math.ceil(10 * c - 1e-9) / 10
        assert printed in (lo, hi), (pair, alpha, c, printed)
        nearest += abs(printed - math.floor(10 * c + 0.5) / 10) < 1e-9
    # every entry but 420 / 78.3 = 5.36 (printed 5.3) is rounded to nearest
    assert nearest == 14


def test_printed_integer_windows_round_down():
    fx = window_fixture()
    assert len(fx["gamma"]) == 6
    for pair, alpha, t_p, t_q, printed in fx["gamma"]:
        assert W.window_size(t_p, t_q, "down") == int(printed), (pair, alpha)


def test_worked_example_of_eq_prefill():
    fx = window_fixture()
    gammas = [W.window_size(t_p, t_q, "nearest") for t_p, t_q, _ in fx["example"]]
    assert gammas == [int(g) for _, _, g in fx["example"]]
    assert gammas[1] / gammas[0] == pytest.approx(fx["window_gain"])


def test_window_rounding_modes_and_clamp():
    assert W.window_size(10, 4, "down") == 2
    assert W.window_size(10, 4, "up") == 3
    assert W.window_size(10, 4, "nearest") == 3      # 2.5 rounds up
    assert W.window_size(0.3, 0.1, "down") == 3     # 2.9999999999999996 snaps to 3
    assert W.window_size(0.3, 0.1, "up") == 3
    assert W.window_size(1, 4, "down") == 1         # c < 1 clamps to 1
    assert W.window_size(1000, 1, "up", gamma_max=16) == 16


def _prefix_len(omega):
    n = 0
    for w in omega:
        if not w:
            break
        n += 1
    return n


def _prob(omega, tau):
    k = sum(omega)
    return tau ** k * (1 - tau) ** (len(omega) - k)


@pytest.mark.parametrize("tau", TAUS)
def test_lemma1_by_enumeration(tau):
    for gamma in range(1, 11):
        ex = sum(_prob(om, tau) * _prefix_len(om)
                 for om in itertools.product((0, 1), repeat=gamma))
        assert W.expected_accepted(tau, gamma) == pytest.approx(ex, rel=1e-12, abs=1e-15)
        # TruncGeo's law: P(X = k) = (1 - tau) tau^k below gamma, tau^gamma at gamma
        for k in range(gamma + 1):
            pk = sum(_prob(om, tau) for om in itertools.product((0, 1), repeat=gamma)
                     if _prefix_len(om) == k)
            want = tau ** gamma if k == gamma else (1 - tau) * tau ** k
            assert pk == pytest.approx(want, rel=1e-12, abs=1e-15)


@pytest.mark.parametrize("tau", TAUS)
def test_two_round_total_by_enumeration(tau):
    # round 2 yields tokens only when round 1 accepted its whole window
    for gamma in range(1, 7):
        tot = 0.0
        for om in itertools.product((0, 1), repeat=2 * gamma):
            x1, x2 = _prefix_len(om[:gamma]), _prefix_len(om[gamma:])
            tot += _prob(om, tau) * (x1 + (x2 if x1 == gamma else 0))
        assert W.expected_total(tau, gamma) == pytest.approx(tot, rel=1e-12, abs=1e-15)


@pytest.mark.parametrize("tau", TAUS)
def test_rollback_speedup_closed_form_at_gamma_eq_c(tau):
    for c in range(1, 13):
        v = W.speedup(c, W.t_psd_rollback(c, tau, c))
        assert v == pytest.approx(0.5 * sum(tau ** k for k in range(1, 2 * c + 1)), rel=1e-12)


def test_practical_reduces_to_ideal_at_full_acceptance():
    for c in (1.0, 1.7, 5.36, 9.0):
        for gamma in range(1, 12):
            assert W.t_sd_practical(c, 1.0, gamma) == pytest.approx(W.t_sd_ideal(c, gamma))
            assert W.t_psd_practical(c, 1.0, gamma) == pytest.approx(W.t_psd_ideal(c, gamma))
        # rollback at tau = 1 and gamma = c is the ideal parallel speedup c
        if c == int(c):
            g = int(c)
            assert W.speedup(c, W.t_psd_rollback(c, 1.0, g)) == pytest.approx(c)


def test_ideal_theorem_values():
    for c in range(1, 12):
        # parallel SD ideal: t for gamma >= c, (c / gamma) t below
        for gamma in range(1, 16):
            want = 1.0 if gamma >= c else c / gamma
            assert W.t_psd_ideal(c, gamma) == pytest.approx(want)
        # at gamma = c the parallel/vanilla speedup ratio is 2c / (c + 1)
        v_sd = W.speedup(c, W.t_sd_ideal(c, c))
        v_psd = W.speedup(c, W.t_psd_ideal(c, c))
        assert v_psd == pytest.approx(c)
        assert v_psd / v_sd == pytest.approx(2 * c / (c + 1))


def test_practical_speedups_and_paravlm_theorem():
    for c in range(1, 10):
        for tau in TAUS:
            v_sd = W.speedup(c, W.t_sd_practical(c, tau, c))
            assert v_sd == pytest.approx(c * (tau * c + 1) / (2 * c))
            v_psd = W.speedup(c, W.t_psd_practical(c, tau, c))
            assert v_psd == pytest.approx(tau * c)
            assert W.paravlm_speedup(tau, c) == pytest.approx(v_psd)
    # the printed gain c*/c with full acceptance: 9/5 = 1.8 and 5/3 = 1.67,
    # printed 1.8 and 1.6 (one decimal, truncated)
    assert math.floor(10 * W.paravlm_speedup(1.0, 9) / W.paravlm_speedup(1.0, 5)) / 10 == 1.8
    assert math.floor(10 * W.paravlm_speedup(1.0, 5) / W.paravlm_speedup(1.0, 3)) / 10 == 1.6


def test_zero_acceptance():
    assert W.expected_accepted(0.0, 5) == 0.0
    assert W.t_psd_practical(4.0, 0.0, 4) == math.inf
    assert W.speedup(4.0, W.t_psd_rollback(4.0, 0.0, 4)) == 0.0
    # vanilla SD still emits the target's own token every round
    assert W.t_sd_practical(4.0, 0.0, 4) == pytest.approx(8.0)


def test_best_window_follows_the_supplement():
    # aggressive window, conservative acceptance (7B/72B, c = 5.36): round down
    assert W.window_size(420, 78.3, "best", tau=0.8) == 5
    # Self-SD, narrow window, high acceptance (7B/7B at alpha 0.5, c = 1.36): round up
    assert W.window_size(78.3, 57.5, "best", tau=0.95) == 2
    # the best window is always the rounded-down or rounded-up ratio
    for t_p, t_q in ((420, 78.3), (420, 57.5), (203, 39.8), (78.3, 46.1), (63.7, 48.2)):
        c = t_p / t_q
        for tau in (0.2, 0.5, 0.7, 0.9, 0.97, 1.0):
            g = W.window_size(t_p, t_q, "best", tau=tau)
            assert g in (math.floor(c), math.ceil(c)), (c, tau, g)
    # below c the speedup still grows, even when by far less than an ulp
    assert W.window_size(1000, 1, "best", tau=0.01, gamma_max=16) == 16
    with pytest.raises(ValueError):
        W.window_size(420, 78.3, "best", tau=0.0)
