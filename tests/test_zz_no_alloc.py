"""GPU: the allocation-free verify entry point, called through the C ABI
(ctypes), against the workspace entry point on the same inputs: two calls in
a row on the same device, the second with a smaller input.  The two share
the kernels, so outputs must be bit-identical."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2603_19610_amd as pv
import workloads as W
from gpu_util import note, to_dev

pytestmark = pytest.mark.gpu


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _noalloc(inp, out, mass, lse, status):
    q = to_dev(inp.q)
    k, v, ctx = to_dev(inp.k), to_dev(inp.v), to_dev(inp.ctx_len)
    B, T, Hq, D = q.shape
    Hkv, n_cap = k.shape[1], k.shape[2]
    st = pv.lib().pvlm_verify_attn_noalloc(
        pv.PVLM_BF16 if q.dtype == torch.bfloat16 else pv.PVLM_F32, B, T, Hq, Hkv, D, n_cap,
        int(inp.ctx_len.max()), float(inp.scale), _ptr(q), _ptr(k), _ptr(v), _ptr(ctx), _ptr(out),
        _ptr(mass), _ptr(lse), _ptr(status), ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    return st, (q, k, v, ctx)


@pytest.mark.parametrize("first,second", [("llava72b", "llava7b"), ("qwen32b", "tiny")])
def test_noalloc_matches_workspace_entry(first, second):
    status = torch.zeros(1, dtype=torch.int32, device="cuda")
    for name in (first, second):      # two calls in a row, the second smaller
        w = W.WORKLOADS[name]
        inp = W.make_verify_inputs(w, layer=1)
        note(f"noalloc verify {name} q{inp.q.shape} k{inp.k.shape}")
        dt = torch.bfloat16 if inp.dtype == "bf16" else torch.float32
        B, T, Hq, D = inp.q.shape
        out = torch.empty((B, T, Hq, D), dtype=dt, device="cuda")
        mass = torch.empty((B, inp.k.shape[2]), dtype=torch.float32, device="cuda")
        lse = torch.empty((B, Hq, T), dtype=torch.float32, device="cuda")
        st, (q, k, v, ctx) = _noalloc(inp, out, mass, lse, status)
        assert st == 0, pv.lib().pvlm_status_string(st)
        ref = pv.verify_attn(q, k, v, ctx, scale=inp.scale, max_ctx=int(inp.ctx_len.max()),
                             ws=pv.Workspace(q.device), status=status)
        torch.cuda.synchronize()
        assert int(status.item()) == 0
        assert torch.equal(out, ref[0]) and torch.equal(mass, ref[1]) and torch.equal(lse, ref[2])


def test_noalloc_rejects_beyond_its_scratch():
    """A shape whose workspace exceeds the fixed scratch is refused before any
    launch (host-side check; nothing runs on the device)."""
    L = pv.lib()
    cap = int(L.pvlm_verify_attn_noalloc_max_bytes())
    B, T, Hq, Hkv, D, n_cap = 16, 9, 64, 8, 128, 1 << 20
    need = int(L.pvlm_verify_attn_workspace_size(pv.PVLM_BF16, B, T, Hq, Hkv, D, n_cap, n_cap - T))
    assert need > cap
    fake = ctypes.c_void_p(0x1000)
    st = L.pvlm_verify_attn_noalloc(pv.PVLM_BF16, B, T, Hq, Hkv, D, n_cap, n_cap - T, 0.088, fake, fake,
                                    fake, fake, fake, None, None, None, None)
    assert st == 4  # PVLM_ERR_WORKSPACE
