"""Seeded synthetic inputs for the ParallelVLM verify + UV-Prune + accept path.

This module is shared by the oracle side (``oracle/``, tests) and the GPU side
(the binding, tests, ``bench.py``).  It holds the workload shapes and the
random draws only: no attention, no similarity, no selection and no
accept/reject arithmetic lives here.  The draft tokens are drawn from the draft
distribution with the Gumbel-max trick, so no softmax is computed either.

Workloads stand in for the paper's video benchmarks (Sec. 5.1 and Suppl. A:
128 frames x 196 tokens, clips over one minute): none of those videos, nor
any model weights, are available, so every tensor is a seeded Gaussian with
the shape, dtype and structure of the corresponding model layer.

Recipe (all draws in float64, then rounded once to the storage dtype):

* Seeds: ``PCG64(SeedSequence([260319610, config_id, layer, tensor_id]))``
  with tensor ids Q=0, K=1, V=2, salient=3, draft logits=4, target noise=5,
  draft tokens=6, uniforms=7, visual hidden=8, text hidden=9, lengths=10,
  page assignment=11.
* Q, K, V ~ N(0, 1).  A fraction of the visual keys is made salient:
  ``k += boost * u_g`` where ``u_g`` is the unit vector of the mean query of
  KV group g (over its query heads and all verify rows), added before RoPE.
* RoPE (rotate-half pairs (i, i + D/2), theta_i = base^(-2i/D)) is applied in
  float64: cache row r sits at position r, verify query t at ctx_len + t.
* Rounding: float64 -> float32 (round to nearest even), then for bf16
  float32 -> bf16 (round to nearest even).  bf16 tensors are stored as
  ``uint16`` bit patterns.
* Cache rows: visual rows [0, m), text rows [m, m + n), then the T = gamma + 1
  verify-block rows [ctx_len, ctx_len + T); rows past that are zero.
* Paged layout: a paged cache holds the same rows as the padded one, in pages
  of P rows (a power of two >= 32) of a shared pool [n_pages][Hkv][P][D].
  Each sequence takes ceil(rows / P) pages; pool pages are handed out in the
  order of a seeded random permutation (so a sequence's pages are scattered
  through the pool), a few spare pool pages stay unused, and page-table
  entries past a sequence's last page are -1.
* Logits: draft ~ N(0, s_d), target = draft + N(0, s_n), float32.  Draft
  tokens are ``argmax(z / temperature + Gumbel)`` per position (the argmax at
  temperature 0).  Uniforms are float64 in [0, 1).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Optional, Tuple

import numpy as np

SEED_ROOT = 260319610

TID_Q, TID_K, TID_V, TID_SAL, TID_DL, TID_TL, TID_TOK, TID_U, TID_HV, TID_HT, TID_LEN, TID_PAGE = \
    range(12)


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    config_id: int
    batch: int
    hq: int
    hkv: int
    head_dim: int
    frames: int
    tokens_per_frame: int
    n_text: int
    gamma: int
    keep_num: int          # keep ratio as an exact fraction keep_num / keep_den
    keep_den: int
    dtype: str             # "f32" or "bf16"
    vocab: int
    salient_frac_num: int  # salient count = floor(m * num / den)
    salient_frac_den: int
    salient_layout: str    # "spread" or "clustered"
    logit_std_draft: float
    logit_std_noise: float
    n_layers: int = 1      # decoder layers of the stacked variant
    crit_layers: int = 1   # L: early layers whose criterion feeds UV-Prune
    ragged_lo: int = 0     # ragged total context lengths (text included), 0 = fixed
    ragged_hi: int = 0
    rope_base: float = 1.0e6
    hidden: int = 0        # hidden size D_h used by the similarity criterion

    @property
    def T(self) -> int:
        return self.gamma + 1

    @property
    def group(self) -> int:
        return self.hq // self.hkv

    @property
    def m_max(self) -> int:
        return self.frames * self.tokens_per_frame

    def lengths(self) -> np.ndarray:
        """Context rows per sequence (visual + text, verify block excluded)."""
        if self.ragged_hi:
            rng = stream(self.config_id, 0, TID_LEN)
            return rng.integers(self.ragged_lo, self.ragged_hi, size=self.batch,
                                endpoint=True).astype(np.int64)
        return np.full(self.batch, self.m_max + self.n_text, dtype=np.int64)

    def m_per_seq(self) -> np.ndarray:
        return self.lengths() - self.n_text

    def keep_count(self, m: np.ndarray) -> np.ndarray:
        return (np.asarray(m, dtype=np.int64) * self.keep_num) // self.keep_den

    def n_cap(self) -> int:
        return int(self.lengths().max()) + self.T


WORKLOADS: Dict[str, Workload] = {
    w.name: w for w in [
        Workload("tiny", 0, 1, 4, 1, 64, 4, 192, 256, 4, 1, 4, "f32", 1024, 2, 100,
                 "spread", 2.0, 0.5, hidden=256),
        Workload("llava7b", 1, 1, 28, 4, 128, 32, 196, 160, 5, 1, 10, "bf16", 152064, 2, 100,
                 "spread", 2.0, 0.5, n_layers=28, crit_layers=20, hidden=3584),
        Workload("llava72b", 2, 1, 64, 8, 128, 64, 196, 256, 8, 1, 10, "bf16", 152064, 2, 100,
                 "spread", 2.0, 0.5, n_layers=80, crit_layers=20, hidden=8192),
        Workload("qwen32b", 3, 4, 40, 8, 128, 128, 256, 512, 8, 1, 20, "bf16", 152064, 1, 100,
                 "clustered", 2.0, 0.5, n_layers=64, crit_layers=20,
                 ragged_lo=16384, ragged_hi=33280, hidden=5120),
        Workload("long", 4, 1, 64, 8, 128, 512, 256, 1024, 16, 3, 100, "bf16", 152064, 2, 100,
                 "spread", 3.0, 1.0, n_layers=80, crit_layers=20, hidden=8192),
    ]
}


def stream(config_id: int, layer: int, tensor_id: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(
        np.random.SeedSequence([SEED_ROOT, int(config_id), int(layer), int(tensor_id)])))


# ---------------------------------------------------------------- rounding --
def f64_to_f32(x: np.ndarray) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bf16 (nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    nan = np.isnan(np.asarray(x, dtype=np.float32))
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)
    r = np.where(nan, np.uint16(0x7FC0), r)
    return r


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    u = (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16)
    return u.view(np.float32).astype(np.float64)


def round_storage(x64: np.ndarray, dtype: str) -> np.ndarray:
    """float64 -> storage array (float32, or uint16 bf16 bits)."""
    f = f64_to_f32(x64)
    if dtype == "f32":
        return f
    if dtype == "bf16":
        return f32_to_bf16_bits(f)
    raise ValueError(dtype)


def storage_to_f64(a: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "f32":
        return np.asarray(a, dtype=np.float32).astype(np.float64)
    if dtype == "bf16":
        return bf16_bits_to_f64(a)
    raise ValueError(dtype)


# -------------------------------------------------------------------- RoPE --
def rope_f64(x: np.ndarray, pos: np.ndarray, base: float) -> np.ndarray:
    """Rotate-half positional rotation of the last axis (size D) in float64.

    ``pos`` broadcasts against ``x[..., 0]``.
    """
    D = x.shape[-1]
    h = D // 2
    theta = base ** (-2.0 * np.arange(h, dtype=np.float64) / D)
    ang = np.asarray(pos, dtype=np.float64)[..., None] * theta
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :h], x[..., h:]
    return np.concatenate([a * c - b * s, a * s + b * c], axis=-1)


# ---------------------------------------------------------- salient tokens --
def salient_rows(w: Workload, b: int, m: int) -> np.ndarray:
    count = (m * w.salient_frac_num) // w.salient_frac_den
    rng = stream(w.config_id, 1000 + b, TID_SAL)
    if count <= 0:
        return np.zeros(0, dtype=np.int64)
    if w.salient_layout == "spread":
        return np.sort(rng.choice(m, size=count, replace=False)).astype(np.int64)
    run = -(-count // 8)
    starts = rng.integers(0, max(1, m - run), size=8)
    rows = np.unique(np.concatenate([np.arange(s, min(m, s + run)) for s in starts]))
    return rows.astype(np.int64)


# ------------------------------------------------------- verify-step inputs --
@dataclasses.dataclass
class VerifyInputs:
    q: np.ndarray        # [B][T][Hq][D] storage dtype
    k: np.ndarray        # [B][Hkv][n_cap][D]
    v: np.ndarray        # [B][Hkv][n_cap][D]
    ctx_len: np.ndarray  # [B] int32 context rows (verify block excluded)
    m: np.ndarray        # [B] int32 visual rows
    n_cap: int
    dtype: str
    scale: float


def make_verify_inputs(w: Workload, layer: int = 1, boost: Optional[float] = None,
                       seed_layer: Optional[int] = None) -> VerifyInputs:
    """One decoder layer of verify inputs.

    For single-layer workloads, ``layer=0`` is the shallow reference layer (same
    base draws, no salient boost) and ``layer=1`` the boosted layer.  For the
    stacked variant pass ``seed_layer=l`` for independent draws per layer.
    The cache is generated one (batch, KV head) slice at a time so the float64
    temporaries stay small.
    """
    lens = w.lengths()
    B, T, Hq, Hkv, D = w.batch, w.T, w.hq, w.hkv, w.head_dim
    n_cap = w.n_cap()
    G = w.group
    sl = 1 if seed_layer is None else seed_layer
    if boost is None:
        boost = 0.0 if layer == 0 else 3.0
    q64 = stream(w.config_id, sl, TID_Q).standard_normal((B, T, Hq, D))
    rk = stream(w.config_id, sl, TID_K)
    rv = stream(w.config_id, sl, TID_V)
    st_dt = np.float32 if w.dtype == "f32" else np.uint16
    k = np.zeros((B, Hkv, n_cap, D), dtype=st_dt)
    v = np.zeros((B, Hkv, n_cap, D), dtype=st_dt)
    for b in range(B):
        N = int(lens[b]) + T
        rows = salient_rows(w, b, int(lens[b]) - w.n_text) if boost else None
        pos = np.arange(N)
        for g in range(Hkv):
            kg = rk.standard_normal((N, D))
            if boost:
                mean_q = q64[b, :, g * G:(g + 1) * G, :].reshape(-1, D).mean(axis=0)
                kg[rows] += boost * (mean_q / np.linalg.norm(mean_q))
            k[b, g, :N] = round_storage(rope_f64(kg, pos, w.rope_base), w.dtype)
            v[b, g, :N] = round_storage(rv.standard_normal((N, D)), w.dtype)
    for b in range(B):
        q64[b] = rope_f64(q64[b], (lens[b] + np.arange(T))[:, None], w.rope_base)
    return VerifyInputs(
        q=round_storage(q64, w.dtype), k=k, v=v, ctx_len=lens.astype(np.int32),
        m=(lens - w.n_text).astype(np.int32), n_cap=n_cap, dtype=w.dtype,
        scale=1.0 / math.sqrt(D))


def random_verify_inputs(B: int, T: int, Hq: int, Hkv: int, D: int, ctx: List[int],
                         dtype: str, seed: int, n_cap: Optional[int] = None,
                         rope_base: float = 1.0e6) -> VerifyInputs:
    """Unstructured verify inputs of an arbitrary shape (for edge cases)."""
    rng = stream(50, seed, TID_Q)
    ctx = np.asarray(ctx, dtype=np.int64)
    n_cap = int(n_cap if n_cap is not None else ctx.max() + T)
    q64 = rng.standard_normal((B, T, Hq, D))
    st_dt = np.float32 if dtype == "f32" else np.uint16
    k = np.zeros((B, Hkv, n_cap, D), dtype=st_dt)
    v = np.zeros((B, Hkv, n_cap, D), dtype=st_dt)
    for b in range(B):
        N = int(ctx[b]) + T
        for g in range(Hkv):
            k[b, g, :N] = round_storage(rope_f64(rng.standard_normal((N, D)), np.arange(N),
                                                 rope_base), dtype)
            v[b, g, :N] = round_storage(rng.standard_normal((N, D)), dtype)
        q64[b] = rope_f64(q64[b], (ctx[b] + np.arange(T))[:, None], rope_base)
    return VerifyInputs(q=round_storage(q64, dtype), k=k, v=v, ctx_len=ctx.astype(np.int32),
                        m=ctx.astype(np.int32), n_cap=n_cap, dtype=dtype,
                        scale=1.0 / math.sqrt(D))


# ------------------------------------------------------------ paged layout --
def page_table(rows, page: int, seed: int = 0, spare: int = 3,
               max_pages: Optional[int] = None) -> Tuple[np.ndarray, int]:
    """Page table for sequences of ``rows[b]`` cache rows in pages of ``page``
    rows.  Returns (table [B][max_pages] int32, n_pages): sequence b's logical
    page j is pool page table[b, j]; entries past its last page are -1."""
    rows = np.asarray(rows, dtype=np.int64)
    need = -(-rows // page)
    mp = int(need.max() if max_pages is None else max_pages)
    if mp < need.max():
        raise ValueError("max_pages too small")
    n_pages = int(need.sum()) + int(spare)
    perm = stream(70, seed, TID_PAGE).permutation(n_pages)
    table = np.full((len(rows), mp), -1, dtype=np.int32)
    o = 0
    for b, nb in enumerate(need):
        table[b, :nb] = perm[o:o + nb]
        o += nb
    return table, n_pages


def to_pages(cache, table: np.ndarray, n_pages: int, page: int):
    """Scatter a padded cache [..., B, Hkv, n_cap, D] (numpy or torch; leading
    layer axes allowed) into a pool [..., n_pages, Hkv, page, D] by ``table``.
    Pool pages that no sequence uses are zero."""
    B, Hkv, n_cap, D = cache.shape[-4:]
    lead = tuple(cache.shape[:-4])
    mp = table.shape[1]
    if n_cap > mp * page:
        raise ValueError("table too short for the cache")
    flat = np.asarray(table).reshape(-1)
    src_sel = np.nonzero(flat >= 0)[0]
    dst_sel = flat[src_sel]
    if isinstance(cache, np.ndarray):
        pad = np.zeros(lead + (B, Hkv, mp * page, D), dtype=cache.dtype)
        pad[..., :n_cap, :] = cache
        pool = np.zeros(lead + (n_pages, Hkv, page, D), dtype=cache.dtype)
    else:
        import torch
        pad = torch.zeros(lead + (B, Hkv, mp * page, D), dtype=cache.dtype, device=cache.device)
        pad[..., :n_cap, :] = cache
        pool = torch.zeros(lead + (n_pages, Hkv, page, D), dtype=cache.dtype,
                           device=cache.device)
        src_sel = torch.from_numpy(src_sel).to(cache.device)
        dst_sel = torch.from_numpy(dst_sel.astype(np.int64)).to(cache.device)
    nl = len(lead)
    blocks = pad.reshape(lead + (B, Hkv, mp, page, D))
    order = tuple(range(nl)) + (nl, nl + 2, nl + 1, nl + 3, nl + 4)
    blocks = blocks.transpose(*order) if isinstance(cache, np.ndarray) else blocks.permute(*order)
    blocks = blocks.reshape(lead + (B * mp, Hkv, page, D))
    pool[..., dst_sel, :, :, :] = blocks[..., src_sel, :, :, :]
    return pool


def crit_boost(w: Workload, layer: int) -> float:
    """Salient boost of decoder layer ``layer`` in the stacked variant."""
    L = max(1, w.crit_layers)
    return 3.0 * min(layer, L) / L


# --------------------------------------------------- similarity criterion --
@dataclasses.dataclass
class HiddenInputs:
    hv: np.ndarray       # [L+1][B][m_cap][Dh] storage dtype
    ht: np.ndarray       # [L+1][B][n_cap][Dh]
    m: np.ndarray        # [B] int32 visual rows
    n: np.ndarray        # [B] int32 text rows
    dtype: str


def make_hidden_inputs(w: Workload, L: int, hidden: Optional[int] = None,
                       m_override: Optional[int] = None,
                       layers: Optional[List[int]] = None) -> HiddenInputs:
    """Layer-wise hidden states of visual and text tokens, layers 0..L.

    Each layer is an independent N(0, 1) draw; salient visual rows gain
    ``3 * l / L`` times the unit mean text direction of layer l.  ``layers``
    restricts which layers are filled (others stay zero) to save memory.
    """
    Dh = hidden or w.hidden
    m_all = w.m_per_seq() if m_override is None else np.full(w.batch, m_override, np.int64)
    n = w.n_text
    m_cap = int(m_all.max())
    hv = np.zeros((L + 1, w.batch, m_cap, Dh))
    ht = np.zeros((L + 1, w.batch, n, Dh))
    for l in range(L + 1):
        if layers is not None and l not in layers:
            continue
        rv = stream(w.config_id, 100 + l, TID_HV)
        rt = stream(w.config_id, 100 + l, TID_HT)
        for b in range(w.batch):
            mb = int(m_all[b])
            hv[l, b, :mb] = rv.standard_normal((mb, Dh))
            ht[l, b] = rt.standard_normal((n, Dh))
            if l > 0 and L > 0:
                d = ht[l, b].mean(axis=0)
                d /= np.linalg.norm(d)
                rows = salient_rows(w, b, mb)
                hv[l, b, rows] += 3.0 * l / L * d
    return HiddenInputs(hv=round_storage(hv, w.dtype), ht=round_storage(ht, w.dtype),
                        m=m_all.astype(np.int32), n=np.full(w.batch, n, np.int32),
                        dtype=w.dtype)


# ------------------------------------------------------- accept inputs --
@dataclasses.dataclass
class AcceptInputs:
    draft_logits: np.ndarray   # [B][gamma][V] float32
    target_logits: np.ndarray  # [B][gamma+1][V] float32
    draft_tokens: np.ndarray   # [B][gamma] int32
    u_accept: np.ndarray       # [B][gamma] float64
    u_sample: np.ndarray       # [B] float64
    temperature: float


def gumbel_tokens(logits: np.ndarray, temperature: float, rng: np.random.Generator) -> np.ndarray:
    """Sample argmax(z / temperature + Gumbel) along the last axis."""
    if temperature == 0.0:
        return np.argmax(logits, axis=-1).astype(np.int32)
    u = rng.random(logits.shape)
    g = -np.log(-np.log(np.maximum(u, 1e-300)))
    return np.argmax(logits.astype(np.float64) / temperature + g, axis=-1).astype(np.int32)


def make_accept_inputs(w: Workload, temperature: float = 1.0, vocab: Optional[int] = None,
                       batch: Optional[int] = None, gamma: Optional[int] = None,
                       salt: int = 0) -> AcceptInputs:
    V = vocab or w.vocab
    B = batch or w.batch
    g = gamma or w.gamma
    dl = stream(w.config_id, salt, TID_DL).standard_normal((B, g + 1, V)) * w.logit_std_draft
    noise = stream(w.config_id, salt, TID_TL).standard_normal((B, g + 1, V)) * w.logit_std_noise
    dl32 = f64_to_f32(dl)
    tl32 = f64_to_f32(dl32.astype(np.float64) + noise)
    draft = np.ascontiguousarray(dl32[:, :g])
    toks = gumbel_tokens(draft, temperature, stream(w.config_id, salt, TID_TOK))
    ru = stream(w.config_id, salt, TID_U)
    return AcceptInputs(draft_logits=draft, target_logits=np.ascontiguousarray(tl32),
                        draft_tokens=toks, u_accept=ru.random((B, g)),
                        u_sample=ru.random(B), temperature=float(temperature))


# --------------------------------------------------------- score inputs --
def make_scores(n_rows: int, m: int, kind: str = "normal", seed: int = 0) -> np.ndarray:
    """float32 score rows for top-k cases: 'normal', 'ties', 'zeros', 'special'."""
    rng = stream(99, seed, TID_U)
    if kind == "normal":
        return rng.standard_normal((n_rows, m)).astype(np.float32)
    if kind == "ties":
        return rng.integers(-3, 4, size=(n_rows, m)).astype(np.float32)
    if kind == "zeros":
        s = np.zeros((n_rows, m), dtype=np.float32)
        s[:, ::2] = -0.0
        return s
    if kind == "special":
        s = rng.integers(-2, 3, size=(n_rows, m)).astype(np.float32)
        sel = rng.random((n_rows, m))
        s[sel < 0.1] = np.nan
        s[(sel >= 0.1) & (sel < 0.15)] = np.inf
        s[(sel >= 0.15) & (sel < 0.2)] = -np.inf
        s[(sel >= 0.2) & (sel < 0.3)] = -0.0
        return s
    raise ValueError(kind)


# ------------------------------------------------- device-side generation --
def make_verify_layer_torch(w: Workload, seed_layer: int, boost: float, device,
                            k_out=None, v_out=None, q_out=None):
    """Same recipe as ``make_verify_inputs`` (N(0,1) draws in float64, salient
    boost along the group's unit mean query before RoPE, rotate-half RoPE in
    float64, rounding to the storage dtype), drawn with torch's generator on
    ``device`` so large stacked caches can be built quickly.  The values differ
    from the numpy stream of the same seed.  Writes into the given tensors
    ([B][Hkv][n_cap][D] and [B][T][Hq][D]) or allocates them.
    """
    import torch
    lens = w.lengths()
    B, T, Hq, Hkv, D = w.batch, w.T, w.hq, w.hkv, w.head_dim
    n_cap = w.n_cap()
    G = w.group
    tdt = torch.float32 if w.dtype == "f32" else torch.bfloat16
    gen = torch.Generator(device=device)
    gen.manual_seed(SEED_ROOT * 1000003 + w.config_id * 10007 + seed_layer)
    if k_out is None:
        k_out = torch.zeros((B, Hkv, n_cap, D), dtype=tdt, device=device)
    if v_out is None:
        v_out = torch.zeros((B, Hkv, n_cap, D), dtype=tdt, device=device)
    if q_out is None:
        q_out = torch.zeros((B, T, Hq, D), dtype=tdt, device=device)
    f64 = torch.float64
    h = D // 2
    theta = w.rope_base ** (-2.0 * torch.arange(h, dtype=f64, device=device) / D)

    def rope(x, pos):
        ang = pos.to(f64)[..., None] * theta
        c, s = torch.cos(ang), torch.sin(ang)
        a, b = x[..., :h], x[..., h:]
        return torch.cat([a * c - b * s, a * s + b * c], dim=-1)

    q64 = torch.randn((B, T, Hq, D), dtype=f64, device=device, generator=gen)
    for b in range(B):
        N = int(lens[b]) + T
        pos = torch.arange(N, device=device)
        rows = None
        if boost:
            rows = torch.from_numpy(salient_rows(w, b, int(lens[b]) - w.n_text)).to(device)
        for g in range(Hkv):
            kg = torch.randn((N, D), dtype=f64, device=device, generator=gen)
            if boost:
                mq = q64[b, :, g * G:(g + 1) * G, :].reshape(-1, D).mean(dim=0)
                kg[rows] += boost * mq / torch.linalg.norm(mq)
            k_out[b, g, :N] = rope(kg, pos).to(torch.float32).to(tdt)
            v_out[b, g, :N] = torch.randn((N, D), dtype=f64, device=device,
                                          generator=gen).to(torch.float32).to(tdt)
        qpos = torch.arange(T, device=device) + int(lens[b])
        q_out[b] = rope(q64[b], qpos[:, None]).to(torch.float32).to(tdt)
    return q_out, k_out, v_out
