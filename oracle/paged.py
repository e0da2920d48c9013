"""Oracle: the verify path over a paged KV cache (float64).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

A paged cache keeps each sequence's rows in fixed-size pages of a pool shared
by the batch: logical row i of sequence b is row i % P of pool page
table[b, i // P] (P rows per page, pool [n_pages][Hkv][P][D]).  The paper does
not fix a cache layout; paging is how a batch of ragged sequences shares one
pool without padding.  The operations are unchanged: verification attention
with the attention mass of attention-guided pruning (Sec. 2.2; Sec. 3,
Challenge 2), the rotation and append of the verify rows, and the compact
draft cache [V*, X] (Sec. 4.2, Stage I).  Every cache row below is read or
written through the table, one row at a time, by ``_row``.

Pins: ``tests/test_oracle_paged.py`` builds pools by scattering a padded cache
into randomly permuted pages and checks these functions against the padded
oracle's results and brute-force rows.
"""
from __future__ import annotations

import numpy as np

from .rope import pair_positions, rotate


def _page_of(table, b, i, P):
    """(pool page, row in page) of logical row i of sequence b."""
    return int(table[b, i // P]), i % P


def _rows(pool, table, b, g, n, P):
    """Logical rows 0 .. n-1 of (b, g), each fetched through the table."""
    out = np.empty((n, pool.shape[-1]), dtype=np.float64)
    for i in range(n):
        pg, r = _page_of(table, b, i, P)
        out[i] = pool[pg, g, r]
    return out


def verify_attn_paged_rows(q, k_pool, v_pool, table, ctx_len, scale, P, rows):
    """Verify attention for the listed (b, h, t) rows over a paged cache.

    q [B][T][Hq][D]; pools [n_pages][Hkv][P][D] (float64 values);
    table [B][max_pages].  Row (b, h, t) sees logical rows
    0 .. ctx_len[b] + t; s_i = scale * <q, k_i>, P_i = softmax(s)_i,
    out = sum_i P_i v_i, lse = log sum_i exp(s_i).
    Returns {(b, h, t): (out[D], lse, P[nvis])}.
    """
    q = np.asarray(q)
    Hq = q.shape[2]
    Hkv = k_pool.shape[1]
    res = {}
    cache = {}
    for (b, h, t) in rows:
        g = (h * Hkv) // Hq
        nvis = int(ctx_len[b]) + t + 1
        key = (b, g)
        if key not in cache or cache[key][0].shape[0] < nvis:
            n_all = int(ctx_len[b]) + q.shape[1]
            cache[key] = (_rows(k_pool, table, b, g, n_all, P),
                          _rows(v_pool, table, b, g, n_all, P))
        kk, vv = cache[key][0][:nvis], cache[key][1][:nvis]
        s = scale * (kk @ np.asarray(q[b, t, h], dtype=np.float64))
        M = s.max()
        e = np.exp(s - M)
        Z = e.sum()
        Pr = e / Z
        res[(b, h, t)] = (Pr @ vv, M + np.log(Z), Pr)
    return res


def verify_attn_paged(q, k_pool, v_pool, table, ctx_len, scale, P):
    """Every row of ``verify_attn_paged_rows``: out [B][T][Hq][D],
    lse [B][Hq][T], mass [B][max_pages * P] (mass[b, i] = sum over heads and
    verify rows of P_i, zero for rows no query sees)."""
    q = np.asarray(q, dtype=np.float64)
    B, T, Hq, D = q.shape
    rows = [(b, h, t) for b in range(B) for h in range(Hq) for t in range(T)]
    r = verify_attn_paged_rows(q, k_pool, v_pool, table, ctx_len, scale, P, rows)
    out = np.zeros((B, T, Hq, D))
    lse = np.zeros((B, Hq, T))
    mass = np.zeros((B, table.shape[1] * P))
    for (b, h, t), (o, l, Pr) in r.items():
        out[b, t, h] = o
        lse[b, h, t] = l
        mass[b, :Pr.shape[0]] += Pr
    return out, lse, mass


def rope_append_paged(q, k_new, v_new, pos, ctx_len, k_pool, v_pool, table, P, base,
                      sections=None):
    """Rotate q and k_new by their positions and write k_new / v_new into a
    copy of the pools at logical rows ctx_len[b] + t, through the table.
    Returns (rotated q, new k pool, new v pool), float64."""
    q = np.asarray(q, dtype=np.float64)
    B, T = q.shape[:2]
    pp = pair_positions(pos, q.shape[-1], sections)
    q_out = rotate(q, pp[:, :, None, :], base)
    k_rot = rotate(np.asarray(k_new, dtype=np.float64), pp[:, :, None, :], base)
    v_new = np.asarray(v_new, dtype=np.float64)
    kp = np.array(k_pool, dtype=np.float64, copy=True)
    vp = np.array(v_pool, dtype=np.float64, copy=True)
    for b in range(B):
        for t in range(T):
            pg, r = _page_of(table, b, int(ctx_len[b]) + t, P)
            kp[pg, :, r, :] = k_rot[b, t]
            vp[pg, :, r, :] = v_new[b, t]
    return q_out, kp, vp


def gather_kv_paged(k_pool, v_pool, table, P, idx, K, tail_begin, tail_len, dst_cap):
    """Compact draft cache from a paged pool: for every layer, batch b and
    KV head g, dst row r < K[b] is logical row idx[b, r], dst row K[b] + r is
    logical row tail_begin[b] + r (r < tail_len[b]); rows past that are 0.
    Pools [n_pages][Hkv][P][D] or [L][n_pages][Hkv][P][D] (one table serves
    every layer); returns [(L,) B][Hkv][dst_cap][D] in the pools' dtype."""
    stacked = k_pool.ndim == 5
    kp = k_pool if stacked else k_pool[None]
    vp = v_pool if stacked else v_pool[None]
    L, _, Hkv, _, D = kp.shape
    B = table.shape[0]
    kd = np.zeros((L, B, Hkv, dst_cap, D), dtype=k_pool.dtype)
    vd = np.zeros((L, B, Hkv, dst_cap, D), dtype=v_pool.dtype)
    for b in range(B):
        src = [int(i) for i in idx[b, :int(K[b])]]
        src += [int(tail_begin[b]) + r for r in range(int(tail_len[b]))]
        for r, i in enumerate(src):
            pg, off = _page_of(table, b, i, P)
            kd[:, b, :, r] = kp[:, pg, :, off]
            vd[:, b, :, r] = vp[:, pg, :, off]
    return (kd, vd) if stacked else (kd[0], vd[0])
