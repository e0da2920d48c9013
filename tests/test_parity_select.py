"""GPU parity: pvlm_topk_select and pvlm_gather_kv, bit-exact against the
oracle (integer selection and byte copies)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2603_19610_amd as pv
import workloads as W
from gpu_util import note, to_dev

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kind", ["normal", "ties", "zeros", "special"])
@pytest.mark.parametrize("m_cap", [1, 1000, 5000, 12544, 16384, 16385, 40000, 131072])
def test_topk_bit_exact(kind, m_cap):
    B = 3
    s = W.make_scores(B, m_cap, kind, seed=m_cap)
    m = np.array([m_cap, max(1, m_cap - 17), max(1, m_cap // 3)], np.int32)
    k = np.array([m[0] // 10, m[1], 0], np.int32)
    k_cap = int(k.max()) + 5
    note(f"topk {kind} m_cap={m_cap}")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx = pv.topk_select(to_dev(s), to_dev(m), to_dev(k), k_cap, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    ref = oracle.topk_select(s, m, k, k_cap)
    assert np.array_equal(idx.cpu().numpy(), ref)


def test_topk_many_long_rows():
    """More rows x slices than compute units: the 256-thread slice path."""
    B, m_cap = 40, 100000
    s = W.make_scores(B, m_cap, "normal", seed=5)
    rng = np.random.default_rng(5)
    m = rng.integers(m_cap // 2, m_cap + 1, size=B).astype(np.int32)
    k = (m // 20).astype(np.int32)
    k_cap = int(k.max())
    note(f"topk many long rows B={B} m_cap={m_cap}")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx = pv.topk_select(to_dev(s), to_dev(m), to_dev(k), k_cap, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert np.array_equal(idx.cpu().numpy(), oracle.topk_select(s, m, k, k_cap))


def test_topk_keep_counts_of_workloads():
    for name in ("tiny", "llava7b", "llava72b", "qwen32b"):
        w = W.WORKLOADS[name]
        m = w.m_per_seq().astype(np.int32)
        k = w.keep_count(m).astype(np.int32)
        s = W.make_scores(w.batch, int(m.max()), "normal", seed=w.config_id)
        note(f"topk workload {name}")
        idx = pv.topk_select(to_dev(s), to_dev(m), to_dev(k), int(k.max()))
        torch.cuda.synchronize()
        assert np.array_equal(idx.cpu().numpy(), oracle.topk_select(s, m, k, int(k.max())))


def test_topk_range_flag():
    s = W.make_scores(1, 100, "normal")
    note("topk k > m flagged")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    idx = pv.topk_select(to_dev(s), to_dev(np.array([50], np.int32)),
                         to_dev(np.array([80], np.int32)), 60, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) & pv.PVLM_DEV_RANGE
    assert np.array_equal(idx.cpu().numpy(), oracle.topk_select(s, [50], [50], 60))


@pytest.mark.parametrize("dt,D", [("bf16", 128), ("bf16", 64), ("f32", 64), ("f32", 128)])
def test_gather_bit_exact(dt, D):
    rng = np.random.default_rng(D)
    B, Hkv, n_cap = 3, 4, 3000
    st = np.uint16 if dt == "bf16" else np.float32
    if dt == "bf16":
        kc = rng.integers(0, 65535, size=(B, Hkv, n_cap, D), dtype=np.uint16)
        vc = rng.integers(0, 65535, size=(B, Hkv, n_cap, D), dtype=np.uint16)
    else:
        kc = rng.standard_normal((B, Hkv, n_cap, D)).astype(st)
        vc = rng.standard_normal((B, Hkv, n_cap, D)).astype(st)
    k = np.array([250, 0, 17], np.int32)
    k_cap = 256
    idx = np.full((B, k_cap), -1, np.int32)
    for b in range(B):
        idx[b, :k[b]] = np.sort(rng.choice(2000, size=k[b], replace=False))
    tb = np.array([2000, 2500, 0], np.int32)
    tl = np.array([256, 500, 5], np.int32)
    dst_cap = 760
    note(f"gather {dt} D={D}")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    kd, vd = pv.gather_kv(to_dev(kc), to_dev(vc), to_dev(idx), to_dev(k), to_dev(tb), to_dev(tl),
                          dst_cap, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    rk, rv = oracle.gather_kv(kc, vc, idx, k, tb, tl, dst_cap)
    gk = kd.cpu().view(torch.int16).numpy().view(np.uint16) if dt == "bf16" else kd.cpu().numpy()
    gv = vd.cpu().view(torch.int16).numpy().view(np.uint16) if dt == "bf16" else vd.cpu().numpy()
    assert np.array_equal(gk.view(np.uint8), rk.view(np.uint8))
    assert np.array_equal(gv.view(np.uint8), rv.view(np.uint8))


def test_gather_rejects_out_of_range_index():
    kc = np.arange(2 * 64 * 128, dtype=np.float32).reshape(1, 2, 64, 128)
    idx = np.array([[3, 70, 5]], np.int32)              # 70 >= n_cap
    note("gather out-of-range index flagged")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    kd, vd = pv.gather_kv(to_dev(kc), to_dev(kc), to_dev(idx), to_dev(np.array([3], np.int32)),
                          to_dev(np.array([60], np.int32)), to_dev(np.array([4], np.int32)), 8,
                          status=status)
    torch.cuda.synchronize()
    assert int(status.item()) & pv.PVLM_DEV_RANGE
    got = kd.cpu().numpy()
    assert np.array_equal(got[0, :, 0], kc[0, :, 3]) and np.all(got[0, :, 1] == 0)
    assert np.array_equal(got[0, :, 3:7], kc[0, :, 60:64])


@pytest.mark.parametrize("m_cap", [1, 1000, 12544, 16385, 40000, 400000])
def test_uvprune_topk_mass_fused(m_cap):
    """pvlm_uvprune_topk_mass equals pvlm_uvprune_score(MASS) followed by
    pvlm_topk_select bit for bit (scores and indices), its scores are within
    one fp32 rounding of the oracle's variation, and its indices are the
    oracle's top-k of those scores.  400000 scores per row take the slice
    path that re-reads the scores every pass."""
    B, L = 3, 4
    rng = np.random.default_rng(m_cap)
    stack = rng.standard_normal((L + 1, B, m_cap)).astype(np.float32)
    stack[:, :, ::7] = stack[:, :, :1]          # repeated values: ties in the scores
    m = np.array([m_cap, max(1, m_cap - 17), max(1, m_cap // 3)], np.int32)
    k = np.array([m[0] // 10, m[1], 0], np.int32)
    k_cap = int(k.max()) + 5
    note(f"uvprune_topk_mass m_cap={m_cap}")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    d_stack, d_m, d_k = to_dev(stack), to_dev(m), to_dev(k)
    score, idx = pv.uvprune_topk_mass(d_stack, d_m, d_k, k_cap, status=status)
    ref_score = pv.uvprune_score_mass(d_stack, d_m, status=status)
    ref_idx = pv.topk_select(ref_score, d_m, d_k, k_cap, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    assert torch.equal(score.view(torch.int32), ref_score.view(torch.int32))
    assert torch.equal(idx, ref_idx)
    s_host = score.cpu().numpy()
    o_score = oracle.uvprune_score_mass(stack.astype(np.float64), m)
    assert np.all(np.abs(s_host - o_score) <= 6e-8 * np.abs(o_score) + 1e-45)
    assert np.array_equal(idx.cpu().numpy(), oracle.topk_select(s_host, m, k, k_cap))
    # without the score output, and with k_cap = 0 (scores only)
    _, idx2 = pv.uvprune_topk_mass(d_stack, d_m, d_k, k_cap, want_score=False)
    s3, _ = pv.uvprune_topk_mass(d_stack, d_m, torch.zeros_like(d_k), 0)
    torch.cuda.synchronize()
    assert torch.equal(idx2, ref_idx)
    assert torch.equal(s3.view(torch.int32), ref_score.view(torch.int32))
