"""Oracle: target verify attention with per-token attention mass (float64).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The target model verifies the gamma drafted tokens in one parallel forward
pass (Sec. 2.2; Sec. 4.2, Parallel Decoding).  Inside each decoder layer,
query t of the verify block (T = gamma + 1 rows: the last accepted token and
the gamma drafts) attends, for every query head h, to all context rows and
causally to the verify-block rows before it.  Grouped-query attention maps
head h to KV head floor(h * Hkv / Hq).  The per-token attention mass is the
attention criterion of attention-guided pruning (Sec. 3, Challenge 2, and the
"attention criterion" ablation in Suppl. D): the normalised probabilities
summed over all heads and verify rows.
"""
from __future__ import annotations

import numpy as np


def verify_attn(q, k, v, ctx_len, scale):
    """Verify attention, log-sum-exp and attention mass, in float64.

    q: [B][T][Hq][D]; k, v: [B][Hkv][n_cap][D] (post-RoPE cache whose rows
    [ctx_len[b], ctx_len[b] + T) are the verify block); ctx_len: [B].
    Returns out [B][T][Hq][D], lse [B][Hq][T], mass [B][n_cap].

    For each (b, h, t): the visible rows are i = 0 .. ctx_len[b] + t;
    s_i = scale * <q, k_i>;  P_i = exp(s_i - M) / sum_j exp(s_j - M) with
    M = max s;  out = sum_i P_i v_i;  lse = M + log(sum_j exp(s_j - M));
    mass[b, i] += P_i.
    """
    q = np.asarray(q, dtype=np.float64)
    k = np.asarray(k, dtype=np.float64)
    v = np.asarray(v, dtype=np.float64)
    B, T, Hq, D = q.shape
    Hkv, n_cap = k.shape[1], k.shape[2]
    out = np.zeros((B, T, Hq, D))
    lse = np.zeros((B, Hq, T))
    mass = np.zeros((B, n_cap))
    for b in range(B):
        for h in range(Hq):
            g = (h * Hkv) // Hq
            for t in range(T):
                nvis = int(ctx_len[b]) + t + 1
                s = scale * (k[b, g, :nvis] @ q[b, t, h])
                M = s.max()
                e = np.exp(s - M)
                Z = e.sum()
                P = e / Z
                out[b, t, h] = P @ v[b, g, :nvis]
                lse[b, h, t] = M + np.log(Z)
                mass[b, :nvis] += P
    return out, lse, mass


def verify_attn_rows(q, k, v, ctx_len, scale, rows):
    """Same definition, evaluated only for the listed (b, h, t) rows.

    Returns {(b, h, t): (out[D], lse, P[nvis])}; used to sample very large
    layers whose full evaluation would take too long on the host.
    """
    q = np.asarray(q)
    B, T, Hq, D = q.shape
    Hkv = k.shape[1]
    res = {}
    for (b, h, t) in rows:
        g = (h * Hkv) // Hq
        nvis = int(ctx_len[b]) + t + 1
        kk = np.asarray(k[b, g, :nvis], dtype=np.float64)
        vv = np.asarray(v[b, g, :nvis], dtype=np.float64)
        s = scale * (kk @ np.asarray(q[b, t, h], dtype=np.float64))
        M = s.max()
        e = np.exp(s - M)
        Z = e.sum()
        P = e / Z
        res[(b, h, t)] = (P @ vv, M + np.log(Z), P)
    return res
