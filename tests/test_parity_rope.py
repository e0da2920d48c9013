"""GPU parity: pvlm_rope_append (1-D RoPE and M-RoPE) against the float64
oracle, and the chain rope_append -> verify_attn against the oracle's chain.

fp32: every element within 2e-6 absolute plus 2e-6 relative (one rounding of
a float64 result; the angle itself is taken in float64).  bf16: within one
bf16 ulp of the oracle's value (one rounding, possibly through fp32).  Value
rows and untouched cache rows: bit-exact.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2603_19610_amd as pv
from gpu_util import assert_lse, assert_mass, assert_out, note, to_host_f64
from oracle import rope as R

pytestmark = pytest.mark.gpu


def _bf16_ulp(x):
    e = np.floor(np.log2(np.maximum(np.abs(x), 1e-30)))
    return 2.0 ** (e - 7)


def _case(dtype, B, T, Hq, Hkv, D, n_cap, ctx, sections, seed, base=1.0e6):
    rng = np.random.default_rng(seed)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    q = torch.from_numpy(rng.standard_normal((B, T, Hq, D)).astype(np.float32)).to(tdt)
    kn = torch.from_numpy(rng.standard_normal((B, T, Hkv, D)).astype(np.float32)).to(tdt)
    vn = torch.from_numpy(rng.standard_normal((B, T, Hkv, D)).astype(np.float32)).to(tdt)
    kc = torch.from_numpy(rng.standard_normal((B, Hkv, n_cap, D)).astype(np.float32)).to(tdt)
    vc = torch.from_numpy(rng.standard_normal((B, Hkv, n_cap, D)).astype(np.float32)).to(tdt)
    ctx = np.asarray(ctx, np.int32)
    if sections is None:
        pos = (ctx[:, None] + np.arange(T)[None, :]).astype(np.int32)
    else:  # visual-style grid positions for the temporal, height and width axes
        t0 = ctx[:, None] + np.arange(T)[None, :]
        pos = np.stack([t0, t0 + rng.integers(0, 40, (B, T)), t0 - rng.integers(0, 40, (B, T))])
        pos = pos.astype(np.int32)
    return q, kn, vn, kc, vc, ctx, pos


def _host(t):
    return t.float().double().numpy()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("sections", [None, (16, 24, 24)])
@pytest.mark.parametrize("shape", [(2, 9, 64, 8, 128, 700, [0, 691]),
                                   (3, 5, 4, 1, 128, 140000, [131072, 7, 139995]),
                                   (1, 17, 40, 8, 128, 33300, [33280])])
def test_rope_append_matches_oracle(dtype, sections, shape):
    B, T, Hq, Hkv, D, n_cap, ctx = shape
    q, kn, vn, kc, vc, ctx, pos = _case(dtype, B, T, Hq, Hkv, D, n_cap, ctx, sections, 7)
    note(f"rope_append {dtype} sections={sections} B={B} T={T} Hq={Hq} Hkv={Hkv} n_cap={n_cap}")
    dev = torch.device("cuda", 0)
    dq, dkn, dvn = q.to(dev), kn.to(dev), vn.to(dev)
    dkc, dvc = kc.to(dev), vc.to(dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    qo = pv.rope_append(dq, dkn, dvn, torch.from_numpy(pos).to(dev),
                        torch.from_numpy(ctx).to(dev), dkc, dvc, base=1.0e6, sections=sections,
                        status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    rq, rk, rv = R.rope_append(_host(q), _host(kn), _host(vn), pos, ctx, _host(kc), _host(vc),
                               1.0e6, sections)
    gq, gk, gv = _host(qo.cpu()), _host(dkc.cpu()), dvc.cpu()
    if dtype == "f32":
        lim_q = 2e-6 + 2e-6 * np.abs(rq)
        lim_k = 2e-6 + 2e-6 * np.abs(rk)
    else:
        lim_q, lim_k = _bf16_ulp(rq) * 1.001, _bf16_ulp(rk) * 1.001
    assert np.all(np.abs(gq - rq) <= lim_q), np.abs(gq - rq).max()
    assert np.all(np.abs(gk - rk) <= lim_k), np.abs(gk - rk).max()
    # value rows are copied and every other row is untouched, bit for bit
    want_v = vc.clone()
    for b in range(B):
        want_v[b, :, ctx[b]:ctx[b] + T] = vn[b].transpose(0, 1)
    assert torch.equal(gv.view(torch.int16 if dtype == "bf16" else torch.int32),
                       want_v.view(torch.int16 if dtype == "bf16" else torch.int32))
    keep = np.ones((B, n_cap), bool)
    for b in range(B):
        keep[b, ctx[b]:ctx[b] + T] = False
    kc_bits = kc.view(torch.int16 if dtype == "bf16" else torch.int32).numpy()
    gk_bits = dkc.cpu().view(torch.int16 if dtype == "bf16" else torch.int32).numpy()
    assert np.array_equal(gk_bits.transpose(0, 2, 1, 3)[keep], kc_bits.transpose(0, 2, 1, 3)[keep])


def test_rope_append_in_place_and_range_flag():
    dev = torch.device("cuda", 0)
    q, kn, vn, kc, vc, ctx, pos = _case("f32", 2, 4, 8, 2, 64, 50, [10, 46], None, 3)
    note("rope_append in place q, ctx clamp")
    dq = q.to(dev)
    ref = pv.rope_append(dq.clone(), kn.to(dev), vn.to(dev), torch.from_numpy(pos).to(dev),
                         torch.from_numpy(ctx).to(dev), kc.to(dev), vc.to(dev), base=1e4)
    out = pv.rope_append(dq, kn.to(dev), vn.to(dev), torch.from_numpy(pos).to(dev),
                         torch.from_numpy(ctx).to(dev), kc.to(dev), vc.to(dev), base=1e4,
                         q_out=dq)
    torch.cuda.synchronize()
    assert out.data_ptr() == dq.data_ptr() and torch.equal(dq, ref)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    bad = torch.tensor([-3, 47], dtype=torch.int32, device=dev)   # 47 + 4 > 50
    dkc = kc.to(dev)
    pv.rope_append(q.to(dev), kn.to(dev), vn.to(dev), torch.from_numpy(pos).to(dev), bad, dkc,
                   vc.to(dev), base=1e4, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) & pv.PVLM_DEV_RANGE


@pytest.mark.parametrize("sections", [None, (8, 12, 12)])
def test_rope_append_then_verify_matches_oracle_chain(sections):
    """The verify step's first two stages: rotate and append the T verify rows,
    then GQA verify attention with the attention mass over the cache."""
    B, T, Hq, Hkv, D, n_cap = 2, 5, 4, 1, 64, 1100
    ctx_np = np.array([1024, 777], np.int32)
    q, kn, vn, kc, vc, ctx, pos = _case("f32", B, T, Hq, Hkv, D, n_cap, ctx_np, sections, 11)
    note(f"rope_append -> verify_attn f32 sections={sections}")
    dev = torch.device("cuda", 0)
    dkc, dvc = kc.to(dev), vc.to(dev)
    dctx = torch.from_numpy(ctx).to(dev)
    qo = pv.rope_append(q.to(dev), kn.to(dev), vn.to(dev), torch.from_numpy(pos).to(dev), dctx,
                        dkc, dvc, base=1.0e6, sections=sections)
    scale = D ** -0.5
    out, mass, lse = pv.verify_attn(qo, dkc, dvc, dctx, scale=scale, max_ctx=int(ctx.max()))
    torch.cuda.synchronize()
    rq, rk, rv = R.rope_append(_host(q), _host(kn), _host(vn), pos, ctx, _host(kc), _host(vc),
                               1.0e6, sections)
    ro, rl, rm = oracle.verify_attn(rq, rk, rv, ctx, scale)
    assert_out(to_host_f64(out), ro)
    assert_lse(to_host_f64(lse), rl)
    assert_mass(to_host_f64(mass), rm, Hq, T)
