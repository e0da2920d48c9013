"""GPU: the co-residency contract of the calls whose workgroups wait on each
other (verify attention, long-row top-k, accept).

Under graph capture those calls are ordinary launches, and the waits of
their workgroups rely on every workgroup becoming resident.  Another
stream's bounded kernels (here GEMMs) can hold compute units for a while;
the waits then last until those kernels retire.  A replay must then give
exactly the eager result, or flag PVLM_DEV_TIMEOUT when a wait gave up: never
a silently wrong result.  Default workspaces are per stream, so calls on two
streams never share counters."""
import numpy as np
import pytest
import torch

import oracle
import paper_2603_19610_amd as pv
import workloads as W
from gpu_util import assert_mass, assert_out, f64, note, to_dev, to_host_f64

pytestmark = pytest.mark.gpu


def test_captured_verify_beside_busy_stream():
    w = W.WORKLOADS["llava72b"]
    inp = W.make_verify_inputs(w, layer=1)
    q, k, v, ctx = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v), to_dev(inp.ctx_len)
    dev = q.device
    note("concurrency: eager reference")
    ref = pv.verify_attn(q, k, v, ctx, ws=pv.Workspace(dev))
    torch.cuda.synchronize()
    out = torch.empty_like(ref[0])
    mass = torch.empty_like(ref[1])
    lse = torch.empty_like(ref[2])
    ws = pv.Workspace(dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    pv.verify_attn(q, k, v, ctx, out=out, mass=mass, lse=lse, ws=ws, status=status)  # sizes ws
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        pv.verify_attn(q, k, v, ctx, out=out, mass=mass, lse=lse, ws=ws, status=status)
    torch.cuda.synchronize()
    other = torch.cuda.Stream()
    a = torch.randn((4096, 4096), device=dev, dtype=torch.bfloat16)
    b = torch.randn((4096, 4096), device=dev, dtype=torch.bfloat16)
    equal = timeouts = 0
    for rep in range(4):
        note(f"concurrency: replay {rep} beside GEMMs on another stream")
        status.zero_()
        out.zero_()
        torch.cuda.synchronize()
        with torch.cuda.stream(other):
            for _ in range(6):
                c = a @ b
        g.replay()                     # no dependency on the other stream
        torch.cuda.synchronize()
        st = int(status.item())
        if st & pv.PVLM_DEV_TIMEOUT:
            timeouts += 1
            ws.buf.zero_()             # counters undefined after a timeout
            torch.cuda.synchronize()
            continue
        assert st == 0, f"device status {st}"
        assert torch.equal(out, ref[0]) and torch.equal(mass, ref[1]) and torch.equal(lse, ref[2])
        equal += 1
    del c
    print(f"[concurrency] {equal} replays equal to eager, {timeouts} flagged a timeout", flush=True)
    assert equal + timeouts == 4


def test_default_workspaces_are_per_stream():
    w = W.WORKLOADS["llava7b"]
    inp = W.make_verify_inputs(w, layer=1)
    q, k, v, ctx = to_dev(inp.q), to_dev(inp.k), to_dev(inp.v), to_dev(inp.ctx_len)
    note("concurrency: default workspaces on two streams")
    ref = pv.verify_attn(q, k, v, ctx, ws=pv.Workspace(q.device))
    torch.cuda.synchronize()
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for s in (s1, s2):
        s.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(s):
            outs.append(pv.verify_attn(q, k, v, ctx))
        torch.cuda.current_stream().wait_stream(s)   # the calls do not overlap
    assert pv.synchronize() == 0
    key = lambda s: ("verify", torch.cuda.current_device(), s.cuda_stream)
    assert pv._ws_cache[key(s1)].buf.data_ptr() != pv._ws_cache[key(s2)].buf.data_ptr()
    for o in outs:
        assert torch.equal(o[0], ref[0]) and torch.equal(o[1], ref[1]) and torch.equal(o[2], ref[2])


@pytest.mark.parametrize("budgets,first", [((224, 32), "72b"), ((128, 128), "72b"), ((224, 32), "wide")])
def test_two_budgeted_streams_run_waiting_calls_together(budgets, first):
    """Verify (72B layer, or 136 rows per KV head over a 20K-token cache, the
    wide variant) on one budgeted stream and verify + accept (7B layer) on
    another, enqueued together and repeated: every result equals the same
    call's result on a lone stream with the same budget, and no wait gives
    up."""
    dev = torch.device("cuda", 0)
    w72, w7 = W.WORKLOADS["llava72b"], W.WORKLOADS["llava7b"]
    if first == "wide":
        a_in = W.random_verify_inputs(1, 17, 64, 8, 128, [20000], "bf16", seed=5)
    else:
        a_in = W.make_verify_inputs(w72, layer=1)
    b_in = W.make_verify_inputs(w7, layer=1)
    A = [to_dev(x) for x in (a_in.q, a_in.k, a_in.v, a_in.ctx_len)]
    Bt = [to_dev(x) for x in (b_in.q, b_in.k, b_in.v, b_in.ctx_len)]
    rng = np.random.default_rng(3)
    Vv, g = 152064, 5
    dl = torch.from_numpy(rng.standard_normal((1, g, Vv)).astype(np.float32)).to(dev)
    tl = torch.from_numpy(rng.standard_normal((1, g + 1, Vv)).astype(np.float32)).to(dev)
    tok = torch.from_numpy(rng.integers(0, Vv, (1, g)).astype(np.int32)).to(dev)
    ua = torch.from_numpy(rng.random((1, g))).to(dev)
    us = torch.from_numpy(rng.random(1)).to(dev)
    s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
    pv.set_stream_cu_budget(s1, budgets[0])
    pv.set_stream_cu_budget(s2, budgets[1])
    ws1, ws2 = pv.Workspace(dev), pv.Workspace(dev)
    st1 = torch.zeros(1, dtype=torch.int32, device=dev)
    st2 = torch.zeros(1, dtype=torch.int32, device=dev)

    def run1():
        return pv.verify_attn(*A, ws=ws1, status=st1)

    def run2():
        o = pv.verify_attn(*Bt, ws=ws2, status=st2)
        n, y, _ = pv.spec_accept(dl, tl, tok, ua, us, 1.0, ws=ws2, status=st2)
        return o + (n, y)

    note(f"budgets {budgets}: each stream alone")
    with torch.cuda.stream(s1):
        r1 = [t.clone() for t in run1()]
    torch.cuda.synchronize()
    with torch.cuda.stream(s2):
        r2 = [t.clone() for t in run2()]
    torch.cuda.synchronize()
    assert int(st1.item()) == 0 and int(st2.item()) == 0
    if first == "wide":
        ro, rl, rm = oracle.verify_attn(f64(a_in.q, "bf16"), f64(a_in.k, "bf16"), f64(a_in.v, "bf16"),
                                        a_in.ctx_len, a_in.scale)
        assert_out(to_host_f64(r1[0]), ro)
        assert_mass(to_host_f64(r1[1]), rm, 64, 17)
    for rep in range(5):
        note(f"budgets {budgets}: both streams together, round {rep}")
        with torch.cuda.stream(s1):
            x1 = run1()
        with torch.cuda.stream(s2):
            x2 = run2()
        torch.cuda.synchronize()
        assert int(st1.item()) == 0 and int(st2.item()) == 0
        assert all(torch.equal(a, b) for a, b in zip(x1, r1))
        assert all(torch.equal(a, b) for a, b in zip(x2, r2))
    pv.set_stream_cu_budget(s1, 0)
    pv.set_stream_cu_budget(s2, 0)
