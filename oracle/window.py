"""Oracle: draft window size and the speedup model of parallel decoding (float64).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Every time is a per-token time in units of t, the draft's single forward time
T_q; the target's verification forward is T_p = c t.  Each function writes out
one statement of the paper:

* ``speed_ratio``            -- Eq. (Prefill): c* = T_p / T_q(alpha).
* ``window_size``            -- Eq. (Prefill) gamma = c*, rounded down, up or to
                                nearest (Suppl. "Window Size Selection"), or the
                                gamma that maximises the rollback speedup.
* ``t_sd_ideal``             -- Suppl. Thm. (Vanilla SD, ideal).
* ``t_psd_ideal``            -- Suppl. Thm. (Parallel SD, ideal).
* ``t_sd_practical``         -- Suppl. Thm. (Vanilla SD, practical).
* ``t_psd_practical``        -- Suppl. Thm. (Parallel SD, practical).
* ``expected_accepted``      -- Suppl. Lemma 1, E[X] of TruncGeo(tau, gamma).
* ``expected_total``         -- the two-round token count in the proof of Suppl.
                                Thm. (Parallel SD with rollback).
* ``t_psd_rollback``         -- Suppl. Thm. (Parallel SD with rollback).
* ``paravlm_speedup``        -- Thm. (paravlm_speedup): tau_hat * c*.
* ``speedup``                -- T_p over a per-token time (speedup against
                                autoregressive decoding with the target).

Readings where the paper is silent or loose:

* X, the accepted length of one window, is the length of the accepted prefix
  (verification stops at the first rejection), so X ~ TruncGeo(tau, gamma):
  P(X = k) = (1 - tau) tau^k for k < gamma and tau^gamma for k = gamma.  The
  rollback proof writes X as the sum of the acceptance indicators; that sum is
  binomial, not TruncGeo, and Lemma 1's mean is the prefix length's.
* At tau = 1 Lemma 1's quotient is 0/0; its limit gamma is used.
* A ratio within 1e-9 (relative) of an integer is taken as that integer before
  rounding, so that T_p / T_q of exact multiples does not round down by one
  ulp.  "nearest" rounds halves up.  gamma is clamped to [1, gamma_max].
* "best" picks, over every integer gamma in [1, gamma_max], the largest
  rollback speedup T_p / T_PSD_r at the (snapped) ratio, the smallest gamma
  on ties.  This is the criterion the supplement names for choosing between
  rounding down and up (the window size against the accepted length).  It
  needs tau > 0.  The comparison is exact (rational arithmetic on the binary
  values of c and tau): at small tau the speedups of successive windows differ
  by less than a float64 ulp, and a rounded comparison would call them tied.
"""
from __future__ import annotations

import math
from fractions import Fraction

SNAP_REL = 1e-9


def speed_ratio(t_p, t_q):
    """Eq. (Prefill): c* = T_p / T_q(alpha)."""
    return float(t_p) / float(t_q)


def t_sd_ideal(c, gamma):
    """Vanilla SD, full acceptance: (gamma T_q + T_p) / (gamma + 1), T_q = 1."""
    t_q, t_p = 1.0, float(c)
    return (gamma * t_q + t_p) / (gamma + 1)


def t_psd_ideal(c, gamma):
    """Parallel SD, full acceptance: max(gamma t, c t) / gamma."""
    return max(gamma * 1.0, float(c)) / gamma


def t_sd_practical(c, tau, gamma):
    """Vanilla SD at acceptance rate tau: (gamma T_q + T_p) / (tau gamma + 1)."""
    t_q, t_p = 1.0, float(c)
    return (gamma * t_q + t_p) / (tau * gamma + 1)


def t_psd_practical(c, tau, gamma):
    """Parallel SD at acceptance rate tau: max(gamma t, c t) / (tau gamma)."""
    den = tau * gamma
    return math.inf if den == 0 else max(gamma * 1.0, float(c)) / den


def expected_accepted(tau, gamma):
    """Lemma 1: E[X] = tau (1 - tau^gamma) / (1 - tau) (limit gamma at tau = 1)."""
    if tau == 1.0:
        return float(gamma)
    return tau * (1.0 - tau ** gamma) / (1.0 - tau)


def expected_total(tau, gamma):
    """Tokens of the two rounds in the rollback proof: (1 + tau^gamma) E[X]."""
    return (1.0 + tau ** gamma) * expected_accepted(tau, gamma)


def t_psd_rollback(c, tau, gamma):
    """Parallel SD with rollback: 2 max(gamma t, c t) / ((1 + tau^gamma) E[X])."""
    den = expected_total(tau, gamma)
    return math.inf if den == 0 else 2.0 * max(gamma * 1.0, float(c)) / den


def speedup(c, per_token_time):
    """Speedup against target-only decoding, T_p / T, with T_p = c t."""
    return 0.0 if per_token_time == math.inf else float(c) / per_token_time


def paravlm_speedup(tau_hat, c_star):
    """Thm. (paravlm_speedup) at gamma = c*: tau_hat gamma T_p / (gamma T_q)."""
    gamma, t_q = float(c_star), 1.0
    t_p = float(c_star) * t_q
    return tau_hat * gamma * t_p / (gamma * t_q)


def _rollback_speedup_exact(c, tau, gamma):
    """T_p / T_PSD_r = c (1 + tau^gamma) E[X] / (2 max(gamma, c)), exactly."""
    c, tau = Fraction(c), Fraction(tau)
    ex = Fraction(gamma) if tau == 1 else tau * (1 - tau ** gamma) / (1 - tau)
    return c * (1 + tau ** gamma) * ex / (2 * max(Fraction(gamma), c))


def _snap(c):
    r = round(c)
    return float(r) if abs(c - r) <= SNAP_REL * abs(c) else c


def window_size(t_p, t_q, rounding="down", tau=None, gamma_max=64):
    """Eq. (Prefill): gamma = c* = T_p / T_q, as an integer in [1, gamma_max]."""
    c = speed_ratio(t_p, t_q)
    cs = _snap(c)
    if rounding == "down":
        g = math.floor(cs)
    elif rounding == "up":
        g = math.ceil(cs)
    elif rounding == "nearest":
        g = math.floor(cs + 0.5)
    elif rounding == "best":
        if tau is None or not 0.0 < tau <= 1.0:
            raise ValueError("best rounding needs 0 < tau <= 1")
        best, g = Fraction(-1), 1
        for cand in range(1, gamma_max + 1):
            v = _rollback_speedup_exact(cs, tau, cand)
            if v > best:
                best, g = v, cand
        return g
    else:
        raise ValueError(rounding)
    return min(max(g, 1), gamma_max)
