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

import paper_2603_19610_amd as pv
import workloads as W
from gpu_util import note, to_dev

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
