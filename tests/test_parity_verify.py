"""GPU parity: pvlm_verify_attn against the float64 oracle (verify attention
output, log-sum-exp and per-token attention mass), element by element."""
import numpy as np
import pytest
import torch

import oracle
import paper_2603_19610_amd as pv
import workloads as W
from gpu_util import (assert_lse, assert_mass, assert_out, f64, note, to_dev, to_host_f64)

pytestmark = pytest.mark.gpu


def _run(inp, max_ctx=None, status=None):
    q, k, v, ctx = (to_dev(inp.q), to_dev(inp.k), to_dev(inp.v), to_dev(inp.ctx_len))
    out, mass, lse = pv.verify_attn(q, k, v, ctx, scale=inp.scale, max_ctx=max_ctx, status=status)
    torch.cuda.synchronize()
    return out, mass, lse


def _check(inp, hq, T, label):
    note(f"verify {label} q{inp.q.shape} k{inp.k.shape} ctx={list(inp.ctx_len)} {inp.dtype}")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    out, mass, lse = _run(inp, status=status)
    assert int(status.item()) == 0
    ro, rl, rm = oracle.verify_attn(f64(inp.q, inp.dtype), f64(inp.k, inp.dtype),
                                    f64(inp.v, inp.dtype), inp.ctx_len, inp.scale)
    assert_out(to_host_f64(out), ro)
    assert_lse(to_host_f64(lse), rl)
    assert_mass(to_host_f64(mass), rm, hq, T)
    return out, mass, lse


SHAPES = [
    # B, T, Hq, Hkv, D, ctx, dtype
    (1, 5, 4, 1, 64, [1024], "f32"),
    (2, 5, 8, 2, 128, [300, 517], "bf16"),        # ragged batch, several tiles
    (1, 6, 28, 4, 128, [700], "bf16"),             # 7B head layout, 3 row tiles
    (1, 9, 64, 8, 128, [1111], "bf16"),            # 72B head layout, 5 row tiles
    (1, 9, 16, 1, 128, [900], "bf16"),             # 144 rows -> two row groups
    (2, 1, 8, 2, 128, [257, 33], "bf16"),          # T = 1 (pre-verify)
    (1, 2, 8, 2, 64, [190], "bf16"),               # D = 64 bf16, T = 2
    (3, 4, 6, 3, 128, [0, 1, 31], "bf16"),         # only the verify block visible
    (1, 3, 8, 8, 128, [20000], "bf16"),            # chunks > 512 tokens: stream variant
    (2, 3, 12, 4, 64, [77, 129], "f32"),           # fp32 path, D = 64, 3 row tiles
    (1, 4, 8, 1, 128, [333], "f32"),               # fp32 path, D = 128
    (1, 32, 16, 2, 128, [700], "bf16"),            # T = 32 (the maximum): 256 rows, 4 row groups
    (4, 9, 28, 4, 128, [100, 900, 3, 1500], "bf16"),  # batch 4 ragged, 7B head layout
    (1, 9, 64, 8, 128, [40000], "bf16"),          # stream variant, 5 row tiles: K/V blocks through LDS
    (1, 8, 64, 8, 128, [30000], "bf16"),          # stream variant, 4 row tiles
    (2, 10, 16, 2, 64, [40000, 25000], "bf16"),   # stream variant, D = 64, 5 row tiles, ragged
    (1, 17, 64, 8, 128, [20000], "bf16"),         # wide variant: 136 rows (9 tiles) in one workgroup
    (1, 12, 64, 8, 128, [24000], "bf16"),         # wide variant, 6 row tiles (3 padding tiles)
    (2, 16, 36, 4, 64, [30000, 9000], "bf16"),    # wide variant, D = 64, 144 rows, empty chunks
    (3, 16, 36, 4, 128, [30000, 5000, 17000], "bf16"),  # wide variant, ragged batch 3: cross-XCD exchanges
]


@pytest.mark.parametrize("shape", SHAPES, ids=lambda s: f"B{s[0]}T{s[1]}H{s[2]}/{s[3]}D{s[4]}{s[6]}")
def test_shapes(shape):
    B, T, Hq, Hkv, D, ctx, dt = shape
    inp = W.random_verify_inputs(B, T, Hq, Hkv, D, ctx, dt, seed=sum(ctx) + Hq)
    _check(inp, Hq, T, "shape")


def test_spare_capacity_and_max_ctx_hint():
    inp = W.random_verify_inputs(2, 5, 8, 2, 128, [400, 250], "bf16", seed=3, n_cap=900)
    note("verify spare capacity n_cap=900")
    ro, rl, rm = oracle.verify_attn(f64(inp.q, "bf16"), f64(inp.k, "bf16"), f64(inp.v, "bf16"),
                                    inp.ctx_len, inp.scale)
    for max_ctx in (None, 400, 600):
        out, mass, lse = _run(inp, max_ctx=max_ctx)
        assert_out(to_host_f64(out), ro)
        assert_mass(to_host_f64(mass), rm, 8, 5)
        assert np.all(to_host_f64(mass)[0, 405:] == 0) and np.all(to_host_f64(mass)[1, 255:] == 0)


def test_device_length_out_of_range_is_flagged_and_clamped():
    inp = W.random_verify_inputs(1, 3, 4, 1, 128, [100], "bf16", seed=4, n_cap=200)
    note("verify ctx_len beyond max_ctx")
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    q, k, v = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v)
    ctx = torch.tensor([150], dtype=torch.int32, device="cuda")   # above max_ctx = 100
    out, mass, lse = pv.verify_attn(q, k, v, ctx, max_ctx=100, status=status)
    torch.cuda.synchronize()
    assert int(status.item()) & pv.PVLM_DEV_RANGE
    ro, _, rm = oracle.verify_attn(f64(inp.q, "bf16"), f64(inp.k, "bf16"), f64(inp.v, "bf16"),
                                   [100], inp.scale)
    assert_out(to_host_f64(out), ro)


@pytest.mark.parametrize("name", ["tiny", "llava7b", "llava72b"])
def test_workload_layers(name):
    w = W.WORKLOADS[name]
    for layer in (0, 1):
        inp = W.make_verify_inputs(w, layer=layer)
        _check(inp, w.hq, w.T, f"{name} layer {layer}")


def test_qwen32b_ragged_batch():
    w = W.WORKLOADS["qwen32b"]
    inp = W.make_verify_inputs(w, layer=1)
    _check(inp, w.hq, w.T, "qwen32b")


def test_long_video_131k():
    w = W.WORKLOADS["long"]
    inp = W.make_verify_inputs(w, layer=1)
    _check(inp, w.hq, w.T, "long")


@pytest.mark.parametrize("shape", [(1, 9, 64, 8, 128, [1111]), (4, 9, 28, 4, 128, [100, 900, 3, 1500]),
                                   (1, 3, 8, 8, 128, [20000]), (1, 17, 64, 8, 128, [20000])],
                         ids=["resident-72B-heads", "resident-ragged-empty-chunks", "stream", "wide"])
def test_without_mass_or_lse(shape):
    """Output alone (no mass, no lse): bit-identical to the full call's output
    (the mass and lse are by-products of the same arithmetic) and within the
    bar against the oracle, after a run in which the later calls' waits would
    hang or time out if an arrival were skipped."""
    B, T, Hq, Hkv, D, ctx = shape
    inp = W.random_verify_inputs(B, T, Hq, Hkv, D, ctx, "bf16", seed=sum(ctx) + 7)
    note(f"verify without mass/lse q{inp.q.shape} k{inp.k.shape} ctx={ctx}")
    q, k, v, c = (to_dev(inp.q), to_dev(inp.k), to_dev(inp.v), to_dev(inp.ctx_len))
    ws = pv.Workspace(torch.device("cuda", 0))
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    full, _, _ = pv.verify_attn(q, k, v, c, scale=inp.scale, ws=ws, status=status)
    outs = []
    for want_mass, want_lse in ((False, False), (True, False), (False, True), (False, False)):
        o, m, l = pv.verify_attn(q, k, v, c, scale=inp.scale, ws=ws, status=status,
                                 want_mass=want_mass, want_lse=want_lse)
        assert (m is None) == (not want_mass) and (l is None) == (not want_lse)
        outs.append(o)
    torch.cuda.synchronize()
    assert int(status.item()) == 0
    for o in outs:
        assert torch.equal(o, full)
    ro, _, _ = oracle.verify_attn(f64(inp.q, "bf16"), f64(inp.k, "bf16"), f64(inp.v, "bf16"),
                                  inp.ctx_len, inp.scale)
    assert_out(to_host_f64(outs[0]), ro)


def test_deterministic_and_reusable_workspace():
    w = W.WORKLOADS["llava72b"]
    inp = W.make_verify_inputs(w, layer=1)
    note("verify 72B determinism x3")
    runs = [_run(inp) for _ in range(3)]
    for o, m, l in runs[1:]:
        assert torch.equal(o, runs[0][0]) and torch.equal(m, runs[0][1]) and torch.equal(l, runs[0][2])
    mass = to_host_f64(runs[0][1])
    assert abs(mass.sum() - w.hq * w.T) < 1e-3 * w.hq * w.T


def test_workspace_reused_across_shapes():
    ws = pv.Workspace(torch.device("cuda", 0))
    shapes = [(2, 5, 8, 2, 128, [300, 517]), (1, 9, 64, 8, 128, [1111]), (1, 17, 64, 8, 128, [20000]),
              (1, 3, 8, 8, 128, [3000]), (3, 4, 6, 3, 128, [0, 1, 31]), (1, 17, 64, 8, 128, [20000]),
              (1, 9, 16, 1, 128, [900])]
    for (B, T, Hq, Hkv, D, ctx) in shapes:
        inp = W.random_verify_inputs(B, T, Hq, Hkv, D, ctx, "bf16", seed=B + T + Hq)
        note(f"verify ws reuse {inp.q.shape} {inp.k.shape}")
        out, mass, lse = pv.verify_attn(to_dev(inp.q), to_dev(inp.k), to_dev(inp.v),
                                        to_dev(inp.ctx_len), ws=ws)
        torch.cuda.synchronize()
        ro, rl, rm = oracle.verify_attn(f64(inp.q, "bf16"), f64(inp.k, "bf16"),
                                        f64(inp.v, "bf16"), inp.ctx_len, inp.scale)
        assert_out(to_host_f64(out), ro)
        assert_mass(to_host_f64(mass), rm, Hq, T)


def test_one_workspace_across_call_kinds():
    """One zero-filled workspace serves verify and accept calls in any order:
    verify's monotonic group counters (same-XCD and cross-XCD exchange
    launches alike) and accept's counters that return to zero share its
    synchronisation region without disturbing each other."""
    ws = pv.Workspace(torch.device("cuda", 0))
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    acc = W.make_accept_inputs(W.WORKLOADS["tiny"], batch=8, salt=11)
    rn, ry, rt = oracle.spec_accept(acc.draft_logits, acc.target_logits, acc.draft_tokens,
                                    acc.u_accept, acc.u_sample, acc.temperature)
    shapes = [(1, 9, 64, 8, 128, [1111]), (1, 6, 28, 4, 128, [700]), (1, 9, 64, 8, 128, [1111]),
              (2, 5, 8, 2, 128, [300, 517]), (1, 6, 28, 4, 128, [700])]
    for i, (B, T, Hq, Hkv, D, ctx) in enumerate(shapes):
        inp = W.random_verify_inputs(B, T, Hq, Hkv, D, ctx, "bf16", seed=40 + i)
        note(f"mixed workspace: verify {inp.q.shape} ctx={ctx}, then accept")
        out, mass, lse = pv.verify_attn(to_dev(inp.q), to_dev(inp.k), to_dev(inp.v),
                                        to_dev(inp.ctx_len), ws=ws, status=status)
        n, y, tie = pv.spec_accept(to_dev(acc.draft_logits), to_dev(acc.target_logits),
                                   to_dev(acc.draft_tokens), to_dev(acc.u_accept),
                                   to_dev(acc.u_sample), acc.temperature, ws=ws, status=status)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        ro, rl, rm = oracle.verify_attn(f64(inp.q, "bf16"), f64(inp.k, "bf16"),
                                        f64(inp.v, "bf16"), inp.ctx_len, inp.scale)
        assert_out(to_host_f64(out), ro)
        assert_lse(to_host_f64(lse), rl)
        assert_mass(to_host_f64(mass), rm, Hq, T)
        ok = rt == 0
        assert np.array_equal(n.cpu().numpy()[ok], rn[ok])
        assert np.array_equal(y.cpu().numpy()[ok], ry[ok])
