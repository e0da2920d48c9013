"""Oracle: Top-K keep and the compact-cache gather.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Eq. (topk_selection) keeps the K visual tokens with the largest UV-Prune
scores, K being the top 1 - alpha fraction of the m visual tokens (Sec. 4.2,
Verifier-Guided Draft Model Pruning).  Readings where the paper is silent:
K = floor(m * keep) in exact integer arithmetic; ties go to the lower token
index; -0.0 ranks equal to +0.0; NaN ranks below every number (-inf
included), lower index first among NaNs; the kept indices are returned in
ascending index order so the compact cache keeps temporal order.

The draft prefills [V*, X] (Sec. 4.2, Stage I): the compact cache holds the
kept visual rows in ascending order followed by the text (tail) rows.
"""
from __future__ import annotations

import numpy as np


def topk_keys(score_row):
    """Sort keys (larger ranks first): float64 values with -0 -> +0, NaN -> below -inf."""
    s = np.asarray(score_row, dtype=np.float64).copy()
    s[s == 0.0] = 0.0          # canonicalise -0.0
    nan = np.isnan(s)
    return s, nan


def topk_select(score, m, k, k_cap):
    """idx [B][k_cap] int32: kept indices ascending, -1 padded.

    The ranking is a full stable sort of the m[b] scores by value descending
    (NaN last) with the lower index first among equals; the first k[b] entries
    are kept.
    """
    score = np.asarray(score)
    B = score.shape[0]
    idx = np.full((B, k_cap), -1, dtype=np.int32)
    for b in range(B):
        mb, kb = int(m[b]), int(k[b])
        vals, nan = topk_keys(score[b, :mb])
        order = sorted(range(mb), key=lambda i: (1 if nan[i] else 0,
                                                 0.0 if nan[i] else -vals[i], i))
        kept = sorted(order[:kb])
        idx[b, :kb] = kept
    return idx


def gather_kv(k_cache, v_cache, idx, K, tail_begin, tail_len, dst_cap):
    """Compact cache rows: dst[b,g,r] = src[b,g,idx[b,r]] for r < K[b], then
    dst[b,g,K[b]+r] = src[b,g,tail_begin[b]+r] for r < tail_len[b].

    Works on any element dtype (bit copy).  Rows past K + tail_len are 0.
    """
    B, Hkv, _, D = k_cache.shape
    kd = np.zeros((B, Hkv, dst_cap, D), dtype=k_cache.dtype)
    vd = np.zeros((B, Hkv, dst_cap, D), dtype=v_cache.dtype)
    for b in range(B):
        rows = [int(i) for i in idx[b, :int(K[b])]]
        rows += [int(tail_begin[b]) + r for r in range(int(tail_len[b]))]
        for r, src in enumerate(rows):
            kd[b, :, r] = k_cache[b, :, src]
            vd[b, :, r] = v_cache[b, :, src]
    return kd, vd
