"""GPU: the whole step captured in a HIP graph replays to the eager results
(several replays with eager work and synchronisation in between), and the
stacked-cache gather equals the per-layer oracle gather."""
import numpy as np
import pytest
import torch

import oracle
import paper_2603_19610_amd as pv
import workloads as W
from gpu_util import note, to_dev

pytestmark = pytest.mark.gpu


def _setup(name):
    w = W.WORKLOADS[name]
    dev = torch.device("cuda", 0)
    inps = [W.make_verify_inputs(w, layer=l) for l in (0, 1)]
    q = [to_dev(i.q) for i in inps]
    k = [to_dev(i.k) for i in inps]
    v = [to_dev(i.v) for i in inps]
    ctx = to_dev(inps[0].ctx_len)
    m = to_dev(w.m_per_seq().astype(np.int32))
    K = to_dev(w.keep_count(w.m_per_seq()).astype(np.int32))
    k_cap = int(K.max())
    n_cap = inps[0].n_cap
    acc = W.make_accept_inputs(w)
    bufs = dict(
        out=torch.empty_like(q[0]), lse=torch.empty((w.batch, w.hq, w.T), device=dev),
        crit=torch.zeros((2, w.batch, n_cap), device=dev),
        score=torch.empty((w.batch, n_cap), device=dev),
        idx=torch.empty((w.batch, k_cap), dtype=torch.int32, device=dev),
        kd=torch.zeros((w.batch, w.hkv, k_cap + w.n_text, w.head_dim), dtype=q[0].dtype, device=dev),
        vd=torch.zeros((w.batch, w.hkv, k_cap + w.n_text, w.head_dim), dtype=q[0].dtype, device=dev),
        na=torch.empty(w.batch, dtype=torch.int32, device=dev),
        nt=torch.empty(w.batch, dtype=torch.int32, device=dev),
        tie=torch.empty(w.batch, dtype=torch.int32, device=dev),
    )
    logits = [to_dev(x) for x in (acc.draft_logits, acc.target_logits, acc.draft_tokens,
                                  acc.u_accept, acc.u_sample)]
    ws_v, ws_a = pv.Workspace(dev), pv.Workspace(dev)

    def step():
        for l in (0, 1):
            pv.verify_attn(q[l], k[l], v[l], ctx, out=bufs["out"], mass=bufs["crit"][l],
                           lse=bufs["lse"], ws=ws_v)
        pv.uvprune_score_mass(bufs["crit"], m, score=bufs["score"])
        pv.topk_select(bufs["score"], m, K, k_cap, idx=bufs["idx"])
        pv.gather_kv(k[1], v[1], bufs["idx"], K, m,
                     torch.full((w.batch,), w.n_text, dtype=torch.int32, device=dev),
                     k_cap + w.n_text, k_dst=bufs["kd"], v_dst=bufs["vd"])
        pv.spec_accept(*logits, acc.temperature, n_accepted=bufs["na"], next_token=bufs["nt"],
                       near_tie=bufs["tie"], ws=ws_a)
    return step, bufs


@pytest.mark.parametrize("name", ["llava72b", "qwen32b"])
def test_graph_replays_match_eager(name):
    note(f"graph capture {name}")
    step, bufs = _setup(name)
    step()
    torch.cuda.synchronize()
    eager = {k: v.clone() for k, v in bufs.items()}
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for rep in range(3):
        for t in bufs.values():
            t.zero_()
        junk = torch.randn(1 << 20, device="cuda").sum()     # eager work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for key, ref in eager.items():
            assert torch.equal(bufs[key], ref), f"replay {rep}: {key} differs from eager"
        del junk


def test_stacked_gather_matches_per_layer():
    rng = np.random.default_rng(9)
    Lyr, B, Hkv, n_cap, D = 5, 2, 3, 700, 128
    kc = rng.integers(0, 65535, size=(Lyr, B, Hkv, n_cap, D), dtype=np.uint16)
    vc = rng.integers(0, 65535, size=(Lyr, B, Hkv, n_cap, D), dtype=np.uint16)
    K = np.array([100, 37], np.int32)
    idx = np.full((B, 128), -1, np.int32)
    for b in range(B):
        idx[b, :K[b]] = np.sort(rng.choice(600, size=K[b], replace=False))
    tb = np.array([600, 610], np.int32)
    tl = np.array([90, 50], np.int32)
    note("stacked gather 5 layers")
    kd, vd = pv.gather_kv(to_dev(kc), to_dev(vc), to_dev(idx), to_dev(K), to_dev(tb), to_dev(tl), 230)
    torch.cuda.synchronize()
    gk = kd.cpu().view(torch.int16).numpy().view(np.uint16)
    gv = vd.cpu().view(torch.int16).numpy().view(np.uint16)
    for l in range(Lyr):
        rk, rv = oracle.gather_kv(kc[l], vc[l], idx, K, tb, tl, 230)
        assert np.array_equal(gk[l], rk) and np.array_equal(gv[l], rv)
