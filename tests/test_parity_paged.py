"""GPU parity of the paged-cache entry points against the paged oracle, which
reads every cache row through the page table.

* pvlm_verify_attn_paged: output, log-sum-exp and attention mass within the
  gates of the padded verify tests; with the same max_ctx it must also equal
  the padded call bit for bit (same launch plan and arithmetic).
* pvlm_rope_append_paged: within the rope tolerances (fp32: 2e-6 abs + rel;
  bf16: one ulp), values and untouched rows bit-exact, and bit-equal to the
  padded call.
* pvlm_gather_kv_paged: bit-exact (pure copy), stacked layers, one table.
Pools come from ``workloads.to_pages``: each sequence's pages scattered over
a seeded random permutation of the pool, a few pool pages unused.
"""
import numpy as np
import pytest
import torch

import oracle
import oracle.paged as OP
import paper_2603_19610_amd as pv
import workloads as W
from gpu_util import assert_lse, assert_mass, assert_out, f64, note, to_dev, to_host_f64

pytestmark = pytest.mark.gpu


def _pages(inp, T, P, seed):
    rows = inp.ctx_len.astype(np.int64) + T
    table, n_pages = W.page_table(rows, P, seed=seed)
    return table, n_pages


def _verify_both(inp, T, P, table, n_pages, status):
    """Padded and paged GPU calls on the same data (paged pools built on the
    device from the padded tensors)."""
    q, k, v, ctx = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v), to_dev(inp.ctx_len)
    max_ctx = int(inp.ctx_len.max())
    out, mass, lse = pv.verify_attn(q, k, v, ctx, scale=inp.scale, max_ctx=max_ctx, status=status)
    kp, vp = W.to_pages(k, table, n_pages, P), W.to_pages(v, table, n_pages, P)
    del k, v
    tab = torch.from_numpy(table).to(q.device)
    pout, pmass, plse = pv.verify_attn_paged(q, kp, vp, tab, ctx, scale=inp.scale, max_ctx=max_ctx,
                                             status=status)
    torch.cuda.synchronize()
    return (out, mass, lse), (pout, pmass, plse)


def _check_paged(inp, Hq, T, P, seed, label, oracle_check=True):
    table, n_pages = _pages(inp, T, P, seed)
    note(f"verify_paged {label} P={P} q{inp.q.shape} ctx={list(inp.ctx_len)} pool={n_pages} pages")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    (out, mass, lse), (pout, pmass, plse) = _verify_both(inp, T, P, table, n_pages, status)
    assert int(status.item()) == 0
    n = mass.shape[1]
    assert torch.equal(out, pout)
    assert torch.equal(lse, plse)
    assert torch.equal(mass, pmass[:, :n])
    assert not pmass[:, n:].any()
    if oracle_check:
        kp = W.to_pages(f64(inp.k, inp.dtype), table, n_pages, P)
        vp = W.to_pages(f64(inp.v, inp.dtype), table, n_pages, P)
        ro, rl, rm = OP.verify_attn_paged(f64(inp.q, inp.dtype), kp, vp, table, inp.ctx_len,
                                          inp.scale, P)
        assert_out(to_host_f64(pout), ro)
        assert_lse(to_host_f64(plse), rl)
        assert_mass(to_host_f64(pmass), rm, Hq, T)


SHAPES = [
    # B, T, Hq, Hkv, D, ctx, P
    (3, 5, 8, 2, 128, [300, 517, 31], 32),         # ragged, sequence shorter than a page
    (2, 9, 64, 8, 128, [1111, 700], 64),           # 72B head layout, 5 row tiles
    (2, 2, 8, 2, 64, [190, 1000], 32),             # D = 64
    (1, 32, 16, 2, 128, [700], 256),               # T = 32, pages larger than a chunk
    (1, 3, 8, 8, 128, [20000], 32),                # chunks > 512 tokens: stream variant
    (2, 9, 64, 8, 128, [40000, 25000], 128),       # stream variant, 5 row tiles, ragged
    (4, 9, 28, 4, 128, [100, 900, 3, 1500], 32),   # batch 4 ragged, empty chunks
    (1, 17, 64, 8, 128, [20000], 32),              # wide variant (136 rows in one workgroup)
]


@pytest.mark.parametrize("shape", SHAPES,
                         ids=lambda s: f"B{s[0]}T{s[1]}H{s[2]}/{s[3]}D{s[4]}P{s[6]}")
def test_verify_paged_shapes(shape):
    B, T, Hq, Hkv, D, ctx, P = shape
    inp = W.random_verify_inputs(B, T, Hq, Hkv, D, ctx, "bf16", seed=sum(ctx) + P)
    _check_paged(inp, Hq, T, P, seed=B + P, label="shape")


def test_verify_paged_qwen32b_ragged_batch():
    """Batch of 4 with lengths drawn from [16384, 33280], 32-row pages (every
    32-token block in its own, scattered page)."""
    w = W.WORKLOADS["qwen32b"]
    inp = W.make_verify_inputs(w, layer=1)
    _check_paged(inp, w.hq, w.T, 32, seed=1, label="qwen32b")


def test_verify_paged_long_131k():
    w = W.WORKLOADS["long"]
    inp = W.make_verify_inputs(w, layer=1)
    _check_paged(inp, w.hq, w.T, 256, seed=2, label="long")


def test_verify_paged_bad_page_entry_is_flagged_and_stays_in_pool():
    inp = W.random_verify_inputs(2, 3, 8, 2, 128, [300, 200], "bf16", seed=9)
    table, n_pages = _pages(inp, 3, 32, seed=3)
    table[1, 2] = n_pages + 7       # outside the pool: read clamped into it, flagged
    note("verify_paged page entry outside the pool")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    q, ctx = to_dev(inp.q), to_dev(inp.ctx_len)
    kp = W.to_pages(to_dev(inp.k), np.where(table < n_pages, table, -1), n_pages, 32)
    vp = W.to_pages(to_dev(inp.v), np.where(table < n_pages, table, -1), n_pages, 32)
    pv.verify_attn_paged(q, kp, vp, torch.from_numpy(table).cuda(), ctx, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) & pv.PVLM_DEV_RANGE


def test_verify_paged_rejects_bad_page_size_and_dtype():
    inp = W.random_verify_inputs(1, 3, 4, 1, 128, [100], "bf16", seed=1)
    q, ctx = to_dev(inp.q), to_dev(inp.ctx_len)
    pool = torch.zeros((8, 1, 48, 128), dtype=torch.bfloat16, device="cuda")
    tab = torch.zeros((1, 3), dtype=torch.int32, device="cuda")
    with pytest.raises(pv.PvlmError):
        pv.verify_attn_paged(q, pool, pool, tab, ctx)
    with pytest.raises((pv.PvlmError, ValueError)):
        pv.verify_attn_paged(q.float(), pool.float(), pool.float(), tab, ctx)


# ------------------------------------------------------------------ gather --
@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_gather_paged_stacked_matches_oracle(dtype):
    L, B, Hkv, D, P = 3, 3, 4, 128, 64
    rng = np.random.default_rng(11)
    rows = np.array([1500, 64, 3000])
    n_cap = int(rows.max())
    st = np.uint16 if dtype == "bf16" else np.float32
    if dtype == "bf16":
        kc = rng.integers(0, 65535, size=(L, B, Hkv, n_cap, D)).astype(st)
        vc = rng.integers(0, 65535, size=(L, B, Hkv, n_cap, D)).astype(st)
    else:
        kc = rng.standard_normal((L, B, Hkv, n_cap, D)).astype(st)
        vc = rng.standard_normal((L, B, Hkv, n_cap, D)).astype(st)
    table, n_pages = W.page_table(rows, P, seed=12)
    K = np.array([300, 0, 700], np.int32)
    k_cap = 800
    idx = np.zeros((B, k_cap), np.int32)
    for b in range(B):
        idx[b, :K[b]] = np.sort(rng.choice(rows[b] - 40, size=K[b], replace=False))
    tb = (rows - 40).astype(np.int32)
    tl = np.full(B, 40, np.int32)
    dst_cap = 760
    kp, vp = W.to_pages(kc, table, n_pages, P), W.to_pages(vc, table, n_pages, P)
    note(f"gather_paged {dtype} L={L} B={B} pool={n_pages}x{P}")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    kd, vd = pv.gather_kv_paged(to_dev(kp), to_dev(vp), to_dev(table), to_dev(idx), to_dev(K),
                                to_dev(tb), to_dev(tl), dst_cap, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    rk, rv = OP.gather_kv_paged(kp, vp, table, P, idx, K, tb, tl, dst_cap)
    view = (lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)) if dtype == "bf16" \
        else (lambda t: t.cpu().numpy())
    assert np.array_equal(view(kd), rk) and np.array_equal(view(vd), rv)
    # the same rows through the padded entry point
    pk, pvv = pv.gather_kv(to_dev(kc), to_dev(vc), to_dev(idx), to_dev(K), to_dev(tb), to_dev(tl),
                           dst_cap)
    bits = (lambda t: t.view(torch.int16)) if dtype == "bf16" else (lambda t: t.view(torch.int32))
    assert torch.equal(bits(kd), bits(pk)) and torch.equal(bits(vd), bits(pvv))


def test_gather_paged_bad_page_entry_skipped_and_flagged():
    B, Hkv, D, P = 1, 2, 128, 32
    rows = np.array([256])
    table, n_pages = W.page_table(rows, P, seed=5)
    table[0, 3] = -5
    kp = torch.randn((n_pages, Hkv, P, D), device="cuda").to(torch.bfloat16)
    idx = torch.arange(0, 256, 2, dtype=torch.int32, device="cuda")[None]
    K = torch.tensor([128], dtype=torch.int32, device="cuda")
    tb = torch.tensor([256], dtype=torch.int32, device="cuda")
    tl = torch.zeros(1, dtype=torch.int32, device="cuda")
    note("gather_paged page entry outside the pool")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    kd, _ = pv.gather_kv_paged(kp, kp, to_dev(table), idx, K, tb, tl, 128, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) & pv.PVLM_DEV_RANGE
    assert not kd[0, :, 48:64].float().any()               # rows of logical page 3 skipped
    assert torch.equal(kd[0, :, :48], kp[table[0, idx[0, :48].cpu().numpy() // P],
                                         :, idx[0, :48].cpu().numpy() % P].transpose(0, 1))


# -------------------------------------------------------------------- rope --
def _bf16_ulp(x):
    e = np.floor(np.log2(np.maximum(np.abs(x), 1e-30)))
    return 2.0 ** (e - 7)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("sections", [None, (16, 24, 24)])
def test_rope_append_paged_matches_oracle(dtype, sections):
    B, T, Hq, Hkv, D, P = 3, 9, 40, 8, 128, 32
    rng = np.random.default_rng(21)
    ctx = np.array([8185, 30, 4100], np.int32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    q = torch.from_numpy(rng.standard_normal((B, T, Hq, D)).astype(np.float32)).to(tdt)
    kn = torch.from_numpy(rng.standard_normal((B, T, Hkv, D)).astype(np.float32)).to(tdt)
    vn = torch.from_numpy(rng.standard_normal((B, T, Hkv, D)).astype(np.float32)).to(tdt)
    table, n_pages = W.page_table(ctx.astype(np.int64) + T, P, seed=8)
    kpool = torch.from_numpy(rng.standard_normal((n_pages, Hkv, P, D)).astype(np.float32)).to(tdt)
    vpool = torch.from_numpy(rng.standard_normal((n_pages, Hkv, P, D)).astype(np.float32)).to(tdt)
    t0 = ctx[:, None] + np.arange(T)[None, :]
    if sections is None:
        pos = t0.astype(np.int32)
    else:
        pos = np.stack([t0, t0 + rng.integers(0, 40, (B, T)), t0 - rng.integers(0, 40, (B, T))])
        pos = pos.astype(np.int32)
    note(f"rope_append_paged {dtype} sections={sections} pool={n_pages}x{P}")
    dev = torch.device("cuda", 0)
    dkp, dvp = kpool.to(dev), vpool.to(dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    qo = pv.rope_append_paged(q.to(dev), kn.to(dev), vn.to(dev), to_dev(pos), to_dev(ctx), dkp, dvp,
                              to_dev(table), base=1.0e6, sections=sections, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    h = lambda t: t.float().double().cpu().numpy()
    rq, rk, rv = OP.rope_append_paged(h(q), h(kn), h(vn), pos, ctx, h(kpool), h(vpool), table, P,
                                      1.0e6, sections)
    gq, gk, gv = h(qo), h(dkp), h(dvp)
    if dtype == "f32":
        for g, r in ((gq, rq), (gk, rk)):
            assert np.all(np.abs(g - r) <= 2e-6 + 2e-6 * np.abs(r))
    else:
        for g, r in ((gq, rq), (gk, rk)):
            assert np.all(np.abs(g - r) <= _bf16_ulp(r) + 1e-30)
    assert np.array_equal(gv, rv)              # values and untouched rows: bit copies
    written = np.zeros(gk.shape, bool)
    for b in range(B):
        for t in range(T):
            i = int(ctx[b]) + t
            written[table[b, i // P], :, i % P] = True
    assert np.array_equal(gk[~written], h(kpool)[~written])


def test_verify_paged_chunk_beyond_the_staged_entries():
    """256 (batch, KV head) groups fill the device, so one chunk spans the
    whole 17,025-row sequence: 533 page entries at 32 rows, more than a
    workgroup stages in LDS, so the kernel reads the table directly.  Bit-equal
    to the padded call; sampled rows against the oracle."""
    B, T, Hq, Hkv, D, ctx, P = 1, 1, 256, 256, 64, 17024, 32
    gen = torch.Generator(device="cuda")
    gen.manual_seed(77)
    q = torch.randn((B, T, Hq, D), device="cuda", generator=gen).to(torch.bfloat16)
    k = torch.randn((B, Hkv, ctx + T, D), device="cuda", generator=gen).to(torch.bfloat16)
    v = torch.randn((B, Hkv, ctx + T, D), device="cuda", generator=gen).to(torch.bfloat16)
    ctx_t = torch.tensor([ctx], dtype=torch.int32, device="cuda")
    table, n_pages = W.page_table(np.array([ctx + T]), P, seed=13)
    assert table.shape[1] > 512
    note(f"verify_paged one chunk of {table.shape[1]} pages (entries read from the table)")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    out, mass, lse = pv.verify_attn(q, k, v, ctx_t, status=status)
    kp, vp = W.to_pages(k, table, n_pages, P), W.to_pages(v, table, n_pages, P)
    pout, pmass, plse = pv.verify_attn_paged(q, kp, vp, torch.from_numpy(table).cuda(), ctx_t,
                                             status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert torch.equal(out, pout) and torch.equal(lse, plse)
    assert torch.equal(mass, pmass[:, :mass.shape[1]])
    rows = [(0, h, 0) for h in (0, 77, 255)]
    heads = sorted({h for _, h, _ in rows})
    ks = k[:, heads].float().double().cpu().numpy()
    vs = v[:, heads].float().double().cpu().numpy()
    qs = q[:, :, heads].float().double().cpu().numpy()
    ref = oracle.verify_attn_rows(qs, ks, vs, np.array([ctx]), D ** -0.5,
                                  [(0, i, 0) for i in range(len(heads))])
    po = to_host_f64(pout)
    for i, h in enumerate(heads):
        o, l, _ = ref[(0, i, 0)]
        assert_out(po[0, 0, h][None], o[None])
        assert abs(float(plse[0, h, 0]) - l) <= 1e-4
