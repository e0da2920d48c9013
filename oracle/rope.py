"""Oracle: rotary position embedding of the verify rows and their append to
the KV cache (float64).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

The verify step (Sec. 2.2; Sec. 4.2, Parallel Decoding) runs the target on
the gamma + 1 speculated positions: their queries and new keys are rotated by
their positions and the new key and value rows join the cache behind the
context, which verify attention then reads.  The targets are LLaVA-OneVision
(Qwen2 language model: 1-D RoPE) and Qwen2.5-VL (multimodal RoPE, "M-RoPE", of
Qwen2-VL, arXiv 2409.12191, Sec. 2.1: each position has a temporal, a height
and a width component, and the frequency pairs are split into three
contiguous sections, one per component).

Definitions written out here (rotate-half pairing, as in RoFormer, arXiv
2104.09864, Sec. 3.4, with the pair (i, i + D/2)):
* frequency of pair i:  w_i = base^(-2 i / D), i = 0 .. D/2 - 1;
* position of pair i:   p (1-D), or p[a(i)] with a(i) = 0 for i < s0, 1 for
                        s0 <= i < s0 + s1, 2 otherwise (M-RoPE, sections
                        (s0, s1, s2), s0 + s1 + s2 = D/2);
* rotation:             (x_i + j x_{i+D/2}) * exp(j p w_i), real part to i,
                        imaginary part to i + D/2 -- written with a complex
                        product.
Values are not rotated.  Key and value rows of verify position t go to cache
row ctx_len[b] + t of their KV head; every other cache row is left as it was.
"""
from __future__ import annotations

import numpy as np


def pair_positions(pos, D, sections=None):
    """Per-pair positions [..., D/2] from 1-D positions [...] or M-RoPE
    positions [3, ...] and the three section widths."""
    half = D // 2
    pos = np.asarray(pos, dtype=np.float64)
    if sections is None:
        return np.repeat(pos[..., None], half, axis=-1)
    s0, s1, s2 = sections
    assert s0 + s1 + s2 == half
    axis = np.array([0] * s0 + [1] * s1 + [2] * s2)
    return np.stack([pos[axis[i]] for i in range(half)], axis=-1)


def rotate(x, pp, base):
    """Rotate x [..., D] by per-pair positions pp [..., D/2] (broadcast over
    heads by the caller)."""
    x = np.asarray(x, dtype=np.float64)
    D = x.shape[-1]
    half = D // 2
    w = base ** (-2.0 * np.arange(half, dtype=np.float64) / D)
    z = (x[..., :half] + 1j * x[..., half:]) * np.exp(1j * pp * w)
    return np.concatenate([z.real, z.imag], axis=-1)


def rope_append(q, k_new, v_new, pos, ctx_len, k_cache, v_cache, base, sections=None):
    """q [B][T][Hq][D], k_new and v_new [B][T][Hkv][D]; pos [B][T] (1-D) or
    [3][B][T] (M-RoPE); caches [B][Hkv][n_cap][D] (copied, not modified).
    Returns (rotated q, new k cache, new v cache), float64."""
    q = np.asarray(q, dtype=np.float64)
    B, T, Hq, D = q.shape
    pp = pair_positions(pos, D, sections)          # [B][T][D/2]
    q_out = rotate(q, pp[:, :, None, :], base)
    k_rot = rotate(k_new, pp[:, :, None, :], base)
    kc = np.array(k_cache, dtype=np.float64, copy=True)
    vc = np.array(v_cache, dtype=np.float64, copy=True)
    v_new = np.asarray(v_new, dtype=np.float64)
    for b in range(B):
        c = int(ctx_len[b])
        for t in range(T):
            kc[b, :, c + t, :] = k_rot[b, t]
            vc[b, :, c + t, :] = v_new[b, t]
    return q_out, kc, vc
