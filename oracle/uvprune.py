"""Oracle: UV-Prune criterion and variation score (float64).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Sec. 4.1 defines the vision-text similarity of visual token V_i and text token
X_j at early layer l as their cosine similarity (Eq. similarity), and the
UV-Prune score of V_i as the change of that similarity between consecutive
layers, summed over all text tokens j = 1..n and layers l = 1..L
(Eq. average_similarity).  Layer 0 is the decoder input.  A zero-norm vector
has cosine 0 with everything (the paper does not say; this is the reading
used throughout).

The same variation operator is applied to a precomputed per-layer criterion
stack c^l_i ("MASS" mode): there the criterion is already summed over the
text side (e.g. the verifier attention mass of layer l), so the score is
sum_{l=1..L} (c^l_i - c^{l-1}_i) (Suppl. D, the attention criterion with variation).

The sums are evaluated literally: no telescoping, no factoring of the j-sum.
"""
from __future__ import annotations

import numpy as np


def cos_similarity(a, b):
    """Eq. (similarity) for two vectors; 0 if either has zero norm."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    na = np.sqrt(np.dot(a, a))
    nb = np.sqrt(np.dot(b, b))
    if na == 0.0 or nb == 0.0:
        return 0.0
    return float(np.dot(a, b) / (na * nb))


def _similarity_matrix(hv, ht):
    """S[i, j] = cos(hv_i, ht_j) for all pairs; explicit loop over text tokens j."""
    hv = np.asarray(hv, dtype=np.float64)
    ht = np.asarray(ht, dtype=np.float64)
    nv = np.sqrt(np.einsum("id,id->i", hv, hv))
    S = np.zeros((hv.shape[0], ht.shape[0]))
    for j in range(ht.shape[0]):
        xj = ht[j]
        nx = np.sqrt(np.dot(xj, xj))
        if nx == 0.0:
            continue
        dots = hv @ xj
        with np.errstate(invalid="ignore", divide="ignore"):
            col = dots / (nv * nx)
        col[nv == 0.0] = 0.0
        S[:, j] = col
    return S


def criterion_cossim(hv, ht, m, n):
    """c[b, i] = sum_{j < n[b]} cos(hv[b, i], ht[b, j]) for i < m[b], one layer.

    hv: [B][m_cap][Dh], ht: [B][n_cap][Dh].  Rows i >= m[b] are 0.
    """
    B, m_cap = hv.shape[0], hv.shape[1]
    c = np.zeros((B, m_cap))
    for b in range(B):
        S = _similarity_matrix(hv[b, :m[b]], ht[b, :n[b]])
        c[b, :m[b]] = S.sum(axis=1)
    return c


def uvprune_score_cossim(hv, ht, m, n):
    """Eq. (average_similarity): sum_j sum_{l=1..L} (S^l_ij - S^{l-1}_ij).

    hv: [L+1][B][m_cap][Dh]; ht: [L+1][B][n_cap][Dh].  Returns [B][m_cap].
    """
    Lp1, B, m_cap = hv.shape[0], hv.shape[1], hv.shape[2]
    score = np.zeros((B, m_cap))
    for b in range(B):
        mb, nb = int(m[b]), int(n[b])
        prev = _similarity_matrix(hv[0, b, :mb], ht[0, b, :nb])
        acc = np.zeros((mb, nb))
        for l in range(1, Lp1):
            cur = _similarity_matrix(hv[l, b, :mb], ht[l, b, :nb])
            acc += cur - prev
            prev = cur
        score[b, :mb] = acc.sum(axis=1)
    return score


def uvprune_score_mass(crit, m):
    """sum_{l=1..L} (c^l_i - c^{l-1}_i) over a criterion stack crit [L+1][B][m_cap]."""
    crit = np.asarray(crit, dtype=np.float64)
    Lp1, B, m_cap = crit.shape
    score = np.zeros((B, m_cap))
    for b in range(B):
        mb = int(m[b])
        acc = np.zeros(mb)
        for l in range(1, Lp1):
            acc += crit[l, b, :mb] - crit[l - 1, b, :mb]
        score[b, :mb] = acc
    return score


# ---- the prefill layer's epilogue (the UV-Prune criterion computed where
#      the layer's hidden states are produced, Sec. 4.1 / 4.2) ---------------
def round_to_storage(x64, dtype):
    """Round float64 values to the storage type: fp32 (round to nearest,
    ties to even), or bf16 through fp32 (round to nearest even on the low 16
    bits of the fp32 pattern).  Returned as float64 values."""
    f = np.asarray(x64, dtype=np.float64).astype(np.float32)
    if dtype == "f32":
        return f.astype(np.float64)
    if dtype != "bf16":
        raise ValueError(dtype)
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16            # (finite values only)
    return r.astype(np.uint32).view(np.float32).astype(np.float64)


def prefill_epilogue(vis_prev, vis_delta, txt_prev, txt_delta, m, n, dtype):
    """The epilogue of a prefill layer with the UV-Prune criterion fused in:
    the residual add h = prev + delta (the sum in fp32, rounded once to the
    storage type) for visual rows i < m[b] and text rows j < n[b], then the
    criterion of the layer, c[b, i] = sum_j cos(h_vis[b, i], h_txt[b, j]),
    over those stored values.  Rows past m[b] / n[b] are left as prev (the
    call does not write them).  Returns (vis_out, txt_out, c), float64."""
    def add(prev, delta, count):
        prev = np.asarray(prev, dtype=np.float64)
        out = prev.copy()
        for b in range(prev.shape[0]):
            k = int(count[b])
            out[b, :k] = round_to_storage(prev[b, :k] + np.asarray(delta, dtype=np.float64)[b, :k], dtype)
        return out
    hv = add(vis_prev, vis_delta, m)
    ht = add(txt_prev, txt_delta, n)
    return hv, ht, criterion_cossim(hv, ht, m, n)
