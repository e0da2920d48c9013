"""Oracle: speculative-sampling accept/reject (float64).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Sec. 2.2: drafted token x_t (t = 1..gamma) is accepted with probability
min(1, p_t(x_t) / q_t(x_t)), where p and q are the target and draft
distributions at that position; at the first rejection a replacement token is
drawn from norm(max(0, p - q)) and the window ends.  Suppl. B: when all gamma
drafts are accepted the target's last verify position yields a bonus token.

Readings where the paper is silent:

* The caller supplies the uniforms: accept iff u_t * q_t(x_t) < p_t(x_t)
  (strict; with q_t(x_t) = 0 this accepts iff p_t(x_t) > 0).
* p = softmax(target_logits / temperature) and likewise q, in float64 with the
  row maximum subtracted first; temperature 0 means greedy: accept iff x_t is
  the target argmax (lowest index on ties) and emit the target argmax.
* Residual / bonus draw by inverse CDF in ascending vocabulary order: the
  emitted token is the smallest y whose cumulative mass exceeds u' * Z, Z the
  total mass.  If rounding leaves no such y, the last y with nonzero mass.
  If the residual has zero total mass, draw from p instead.
* A decision is a near tie when |u q - p| <= 1e-9 max(p, u q), and a draw is a
  near tie when u' Z lies within 1e-9 Z of a CDF boundary of the emitted
  token (the lower boundary of token 0 is an exact 0 and never counts); near
  ties are reported so a comparison can skip them.
"""
from __future__ import annotations

import numpy as np

NEAR_TIE_REL = 1e-9


def softmax_t(z, temperature):
    """softmax(z / temperature) in float64 with the maximum subtracted first."""
    z = np.asarray(z, dtype=np.float64)
    M = z.max()
    e = np.exp((z - M) / temperature)
    return e / e.sum()


def _inverse_cdf(r, u):
    cum = np.cumsum(r)
    Z = cum[-1]
    thr = u * Z
    hits = np.nonzero(cum > thr)[0]
    if hits.size:
        y = int(hits[0])
    else:
        y = int(np.nonzero(r > 0)[0][-1])
    near = abs(cum[y] - thr) <= NEAR_TIE_REL * Z
    if y > 0:
        near = near or abs(cum[y - 1] - thr) <= NEAR_TIE_REL * Z
    return y, near


def spec_accept(draft_logits, target_logits, draft_tokens, u_accept, u_sample, temperature):
    """Returns (n_accepted [B] int32, next_token [B] int32, near_tie [B] int32)."""
    dl = np.asarray(draft_logits)
    tl = np.asarray(target_logits)
    B, gamma, V = dl.shape
    tau = float(np.float32(temperature))
    n_acc = np.zeros(B, dtype=np.int32)
    nxt = np.zeros(B, dtype=np.int32)
    near = np.zeros(B, dtype=np.int32)
    for b in range(B):
        if tau == 0.0:
            a = gamma
            for t in range(gamma):
                if int(draft_tokens[b, t]) != int(np.argmax(tl[b, t])):
                    a = t
                    break
            n_acc[b] = a
            nxt[b] = int(np.argmax(tl[b, a]))
            continue
        a = gamma
        tie = False
        for t in range(gamma):
            p = softmax_t(tl[b, t], tau)
            q = softmax_t(dl[b, t], tau)
            x = int(draft_tokens[b, t])
            lhs = float(u_accept[b, t]) * q[x]
            rhs = p[x]
            if abs(lhs - rhs) <= NEAR_TIE_REL * max(lhs, rhs):
                tie = True
            if not lhs < rhs:
                a = t
                break
        p = softmax_t(tl[b, a], tau)
        if a < gamma:
            r = np.maximum(0.0, p - softmax_t(dl[b, a], tau))
            if r.sum() == 0.0:
                r = p
        else:
            r = p
        y, tie_draw = _inverse_cdf(r, float(u_sample[b]))
        n_acc[b] = a
        nxt[b] = y
        near[b] = int(tie or tie_draw)
    return n_acc, nxt, near
