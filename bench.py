"""Benchmark of the ParallelVLM verify + UV-Prune + gather + accept step on one MI355X.

Workload (default): the LLaVA-OneVision-72B decode step, stacked over all 80
decoder layers: each layer's verify attention (64 query / 8 KV heads, head dim
128, 12544 visual + 256 text cache rows, gamma = 8 so 9 verify rows) with the
fused attention mass; after the last early layer (L = 20) the UV-Prune score
over the layer 0..20 masses and the top-10% keep; the kept rows plus the text
rows of all 80 layers gathered into the draft's compact cache; and the
speculative accept/reject over a 152064-token vocabulary.  Inputs are seeded
synthetic tensors resident in HBM before timing starts.  The step runs as one
HIP graph replay (falls back to eager launches if capture fails).

Prints ONE JSON line.  `value` is microseconds per decoder layer (step time /
80); `achieved_hbm_tbs` is algorithmic bytes / step time.  `roofline` covers the
dominant kernel (verify attention): its mean launch duration comes from HIP
events around replays of a graph of 80 verify launches on the replaying stream.  `cpu_baseline` times the float64 oracle on the host for
a bounded sample of the same step.

    python bench.py [--gpus 1] [--steps 20] [--warmup 5] [--mode stacked|layer]
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "verify+prune step us/layer & achieved HBM TB/s, LLaVA-OV-72B layer shape"
HBM_PEAK_GBS = 8000.0
PROFILES = os.path.join(ROOT, "profiles")
VERIFY_SRCS = [os.path.join(ROOT, "paper_2603_19610_amd", "csrc", f)
               for f in ("verify_attn.hip", "common.h")]
COPY_BYTES = 512 << 20


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="llava72b")
    ap.add_argument("--mode", choices=["stacked", "layer"], default="stacked")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernel-reps", type=int, default=80,
                    help="verify launches per graph replay timed for the roofline")
    ap.add_argument("--verify-only", type=int, default=0,
                    help="profiling helper: run N verify launches and exit")
    ap.add_argument("--copy-only", type=int, default=0,
                    help="profiling helper: N device copies of 512 MiB (counter calibration)")
    return ap.parse_args()


# ------------------------------------------------------------ byte counts --
def verify_bytes(w, esize=2):
    """Algorithmic HBM bytes of one verify launch: K and V of the N + T visible
    rows, Q, O, mass and lse, each moved once."""
    N = int(w.lengths().sum()) + w.batch * w.T
    kv = 2 * N * w.hkv * w.head_dim * esize
    qo = 2 * w.batch * w.T * w.hq * w.head_dim * esize
    return kv + qo + 4 * w.batch * w.n_cap() + 4 * w.batch * w.hq * w.T


def gather_bytes(w, esize=2):
    m = w.m_per_seq()
    rows = int((w.keep_count(m) + w.n_text).sum())
    return 2 * 2 * rows * w.hkv * w.head_dim * esize + 4 * int(w.keep_count(m).sum())


def uvprune_bytes(w):
    m = int(w.m_per_seq().sum())
    return 3 * 4 * m          # read c^0 and c^L, write the score


def topk_bytes(w):
    m = w.m_per_seq()
    return 4 * int(m.sum()) + 4 * int(w.keep_count(m).sum())


def accept_bytes(w):
    return 4 * w.batch * (2 * w.gamma + 1) * w.vocab


# ---------------------------------------------------------------- traffic --
def measured_traffic():
    """HBM bytes per verify launch from the committed rocprofv3 counter runs,
    or None when the kernel source changed since they were taken."""
    path = os.path.join(PROFILES, "verify_attn_llava72b_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    h = re.search(r"kernel source sha256 \(verify_attn\.hip \+ common\.h\): ([0-9a-f]{64})", text)
    t = re.search(r"traffic_bytes_per_launch: ([0-9.eE+]+)", text)
    if not h or not t:
        return None
    cur = hashlib.sha256()
    for f in VERIFY_SRCS:
        cur.update(open(f, "rb").read())
    return float(t.group(1)) if cur.hexdigest() == h.group(1) else None


# ------------------------------------------------------------ CPU baseline --
def cpu_baseline(w, layers_host, crit_layers, per_layer_ok):
    """Time the float64 oracle on host copies of the same inputs."""
    import oracle
    import workloads as W
    from threadpoolctl import threadpool_info, threadpool_limits

    cores = len(os.sched_getaffinity(0))
    with threadpool_limits(limits=cores):
        blas = [i.get("num_threads", 1) for i in threadpool_info()]
        threads = max(blas) if blas else 1
        t_verify = []
        masses = []
        for (q, k, v, ctx) in layers_host:
            t0 = time.perf_counter()
            _, _, mass = oracle.verify_attn(q, k, v, ctx, 1.0 / np.sqrt(w.head_dim))
            t_verify.append(time.perf_counter() - t0)
            masses.append(mass)
        m = w.m_per_seq().astype(np.int32)
        K = w.keep_count(m).astype(np.int32)
        stack = np.stack([masses[i % len(masses)] for i in range(crit_layers + 1)])
        t0 = time.perf_counter()
        score = oracle.uvprune_score_mass(stack, m)
        t_uv = time.perf_counter() - t0
        t0 = time.perf_counter()
        idx = oracle.topk_select(score, m, K, int(K.max()))
        t_topk = time.perf_counter() - t0
        q, k, v, ctx = layers_host[0]
        t0 = time.perf_counter()
        oracle.gather_kv(k, v, idx, K, m, np.full(w.batch, w.n_text), int(K.max()) + w.n_text)
        t_gather = time.perf_counter() - t0
        acc = W.make_accept_inputs(w)
        t0 = time.perf_counter()
        oracle.spec_accept(acc.draft_logits, acc.target_logits, acc.draft_tokens, acc.u_accept,
                           acc.u_sample, acc.temperature)
        t_acc = time.perf_counter() - t0
    per_layer = np.mean(t_verify) + t_gather
    once = t_uv + t_topk + t_acc
    L = per_layer_ok
    us_per_layer = (per_layer + once / L) * 1e6
    return {
        "value": round(us_per_layer, 1), "unit": "us/layer", "cores": int(threads),
        "kind": "oracle",
        "sample": (f"float64 oracle on {len(layers_host)} of the {L} layers' verify inputs "
                   f"(mean {np.mean(t_verify):.2f} s/layer), gather of one layer "
                   f"({t_gather:.3f} s), UV-Prune over {crit_layers + 1} masses ({t_uv:.3f} s), "
                   f"top-k ({t_topk:.3f} s) and accept ({t_acc:.3f} s); per layer = verify + "
                   f"gather + (UV-Prune + top-k + accept) / {L}; host cores available {cores}"),
    }


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: this build has no multi-GPU path (the hot path "
              "runs on one MI355X; see DESIGN.md for how it would shard). Run with --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2603_19610_amd as pv
    import workloads as W

    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.copy_only:  # a plain copy of known size: 512 MiB read + 512 MiB written
        src = torch.ones(COPY_BYTES // 2, dtype=torch.bfloat16, device=dev)
        dst = torch.empty_like(src)
        for _ in range(args.copy_only):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_only": args.copy_only, "bytes_read": COPY_BYTES,
                          "bytes_written": COPY_BYTES}))
        return
    w = W.WORKLOADS[args.workload]
    stacked = args.mode == "stacked"
    NL = w.n_layers if stacked else 1
    L = w.crit_layers if stacked else 1
    B, T, Hq, Hkv, D = w.batch, w.T, w.hq, w.hkv, w.head_dim
    n_cap = w.n_cap()
    lens = w.lengths()
    m_np = w.m_per_seq().astype(np.int32)
    K_np = w.keep_count(m_np).astype(np.int32)
    k_cap = int(K_np.max())
    dst_cap = k_cap + w.n_text

    # ---- inputs resident in HBM
    t0 = time.time()
    tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    Kc = torch.zeros((NL, B, Hkv, n_cap, D), dtype=tdt, device=dev)
    Vc = torch.zeros_like(Kc)
    Q = torch.zeros((NL, B, T, Hq, D), dtype=tdt, device=dev)
    for l in range(NL):
        layer_id = l if stacked else 1
        W.make_verify_layer_torch(w, layer_id, W.crit_boost(w, layer_id), dev,
                                  k_out=Kc[l], v_out=Vc[l], q_out=Q[l])
    q0 = k0 = v0 = None
    if not stacked:  # layer 0 = the same draws without the salient boost
        q0, k0, v0 = W.make_verify_layer_torch(w, 1, 0.0, dev)
    torch.cuda.synchronize()
    log(f"inputs: {NL} layer(s), cache {2 * Kc.numel() * Kc.element_size() / 1e9:.2f} GB, "
        f"{time.time() - t0:.1f} s")
    ctx = torch.from_numpy(lens.astype(np.int32)).to(dev)
    m_t = torch.from_numpy(m_np).to(dev)
    k_t = torch.from_numpy(K_np).to(dev)
    tail_b = m_t.clone()
    tail_l = torch.full((B,), w.n_text, dtype=torch.int32, device=dev)
    acc = W.make_accept_inputs(w)
    dl = torch.from_numpy(acc.draft_logits).to(dev)
    tl = torch.from_numpy(acc.target_logits).to(dev)
    tok = torch.from_numpy(acc.draft_tokens).to(dev)
    ua = torch.from_numpy(acc.u_accept).to(dev)
    us = torch.from_numpy(acc.u_sample).to(dev)

    out = torch.empty((B, T, Hq, D), dtype=tdt, device=dev)
    lse = torch.empty((B, Hq, T), dtype=torch.float32, device=dev)
    crit = torch.zeros((L + 1, B, n_cap), dtype=torch.float32, device=dev)
    mass_x = torch.empty((B, n_cap), dtype=torch.float32, device=dev)
    score = torch.empty((B, n_cap), dtype=torch.float32, device=dev)
    idx = torch.empty((B, k_cap), dtype=torch.int32, device=dev)
    kd = torch.zeros((NL, B, Hkv, dst_cap, D), dtype=tdt, device=dev)
    vd = torch.zeros_like(kd)
    na = torch.empty(B, dtype=torch.int32, device=dev)
    nt = torch.empty(B, dtype=torch.int32, device=dev)
    tie = torch.empty(B, dtype=torch.int32, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    ws_v = pv.Workspace(dev)
    ws_a = pv.Workspace(dev)
    max_ctx = int(lens.max())

    if not stacked:  # the shallow reference layer's mass exists before the step
        pv.verify_attn(q0, k0, v0, ctx, max_ctx=max_ctx, out=out, mass=crit[0], lse=lse, ws=ws_v,
                       status=status)

    def verify(l, mass):
        pv.verify_attn(Q[l], Kc[l], Vc[l], ctx, max_ctx=max_ctx, out=out, mass=mass, lse=lse,
                       ws=ws_v, status=status)

    def step():
        for l in range(NL):
            if stacked:
                verify(l, crit[l] if l <= L else mass_x)
            else:
                verify(0, crit[1])
            if l == (L if stacked else 0):
                pv.uvprune_score_mass(crit, m_t, score=score, status=status)
                pv.topk_select(score, m_t, k_t, k_cap, idx=idx, status=status)
        pv.gather_kv(Kc, Vc, idx, k_t, tail_b, tail_l, dst_cap, k_dst=kd, v_dst=vd, status=status)
        pv.spec_accept(dl, tl, tok, ua, us, acc.temperature, n_accepted=na, next_token=nt,
                       near_tie=tie, ws=ws_a, status=status)

    if args.verify_only:
        for r in range(args.verify_only):
            verify(r % NL, mass_x)
        torch.cuda.synchronize()
        print(json.dumps({"verify_only": args.verify_only, "status": int(status.item())}))
        return

    # eager warm-up (also sizes the workspaces before any capture)
    step()
    torch.cuda.synchronize()
    run = step
    graph_used = False
    if not args.no_graph:
        try:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(s):
                step()
            torch.cuda.current_stream().wait_stream(s)
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                step()
            torch.cuda.synchronize()
            run = g.replay
            graph_used = True
        except Exception as e:  # capture unsupported: time eager launches
            log(f"graph capture failed ({type(e).__name__}: {e}); timing eager launches")
            torch.cuda.synchronize()
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    status.zero_()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    h0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        run()
    e1.record()
    torch.cuda.synchronize()
    host_s = time.perf_counter() - h0
    ms_step = e0.elapsed_time(e1) / args.steps
    st = int(status.item())
    if st:
        log(f"device status {st} during the timed steps")

    # ---- dominant kernel: verify attention.  `reps` launches (cycling over
    # the layers) captured in one graph; events on the replaying stream around
    # whole replays give the mean launch duration, inter-kernel gaps included.
    reps = args.kernel_reps
    vb = verify_bytes(w)
    k_mean = None
    if graph_used:
        gv = torch.cuda.CUDAGraph()
        with torch.cuda.graph(gv):
            for r in range(reps):
                verify((7 * r + 3) % NL, mass_x)
        gv.replay()
        torch.cuda.synchronize()
        n_rep = 5
        a_ev = torch.cuda.Event(enable_timing=True)
        b_ev = torch.cuda.Event(enable_timing=True)
        a_ev.record()
        for _ in range(n_rep):
            gv.replay()
        b_ev.record()
        torch.cuda.synchronize()
        k_mean = a_ev.elapsed_time(b_ev) * 1e3 / (n_rep * reps)
    # one eager (cooperative) launch at a time behind a busy stream: the
    # per-launch cost a caller outside a graph sees
    blocker = torch.randn((4096, 4096), device=dev, dtype=torch.bfloat16)
    n_eager = 40
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(n_eager)]
    torch.cuda.synchronize()
    for _ in range(48):         # keep the GPU busy while the launches are enqueued
        blocker = blocker @ blocker
        blocker = blocker / blocker.abs().max()
    for r in range(n_eager):
        a, b = evs[r]
        a.record()
        verify((7 * r + 3) % NL, mass_x)
        b.record()
    torch.cuda.synchronize()
    eager_us = float(np.mean([a.elapsed_time(b) * 1e3 for a, b in evs][2:]))
    if k_mean is None:
        k_mean = eager_us
    achieved = vb / (k_mean * 1e-6) / 1e9

    step_bytes = NL * (verify_bytes(w) + gather_bytes(w)) + uvprune_bytes(w) + topk_bytes(w) \
        + accept_bytes(w)
    us_layer = ms_step * 1e3 / NL
    traffic = measured_traffic()

    cpu = None
    if not args.no_cpu_baseline:
        hosts = []
        sample = [1, 2] if not stacked else [0, 20, 40, 79]
        for l in sample[:4]:
            li = min(l, NL - 1)
            hosts.append((W.storage_to_f64(Q[li].float().cpu().numpy(), "f32"),
                          Kc[li].float().cpu().double().numpy(),
                          Vc[li].float().cpu().double().numpy(), lens))
        t0 = time.time()
        cpu = cpu_baseline(w, hosts, L, NL)
        log(f"cpu baseline {time.time() - t0:.1f} s")

    rec = {
        "metric": METRIC,
        "value": round(us_layer, 3),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}-{'stacked-%dL' % NL if stacked else 'single-layer'}",
            "batch": B, "query_heads": Hq, "kv_heads": Hkv, "head_dim": D,
            "visual_tokens": int(m_np.max()), "text_tokens": w.n_text, "gamma": w.gamma,
            "verify_rows": T, "keep": f"{w.keep_num}/{w.keep_den}", "uvprune_layers": L,
            "vocab": w.vocab, "layers": NL, "criterion": "attention mass",
            "hip_graph": graph_used,
        },
        "achieved_hbm_tbs": round(step_bytes / (ms_step * 1e-3) / 1e12, 3),
        "step_bytes": step_bytes,
        "host_ms_per_step": round(host_s * 1e3 / args.steps, 4),
        "roofline": {
            "bound": "hbm", "kernel": "verify_mfma_kernel<128,5,resident>",
            "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "bytes_per_launch": vb, "launch_us": round(k_mean, 3),
            "launch_timing": ("graph of %d launches, events around replays" % reps
                              if graph_used else "eager launches, events around each"),
            "eager_launch_us": round(eager_us, 3),
        },
        "cpu_baseline": cpu,
        "device_status": st,
    }
    print(json.dumps(rec))


if __name__ == "__main__":
    main()
