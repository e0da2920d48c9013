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
events around replays of a graph of 80 verify launches on the replaying stream.
`stages_us` times each stage the same way; `copy_gbs` is the device-to-device
copy bandwidth measured in the same run; `other_configs` times the single-layer
step of the other model shapes; `cossim` times the similarity criterion.
`cpu_baseline` times the float64 oracle on the host for a bounded sample of the
same step.

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
OTHER_CONFIGS = ("tiny", "llava7b", "llava72b", "qwen32b", "long")


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
    ap.add_argument("--no-extra", action="store_true",
                    help="skip the other model shapes and the similarity criterion")
    ap.add_argument("--kernel-reps", type=int, default=80,
                    help="verify launches per graph replay timed for the roofline")
    ap.add_argument("--verify-only", type=int, default=0,
                    help="profiling helper: run N verify launches and exit")
    ap.add_argument("--gather-only", type=int, default=0,
                    help="profiling helper: one eager step, then N 80-layer gathers, and exit")
    ap.add_argument("--copy-only", type=int, default=0,
                    help="profiling helper: N device copies of 512 MiB (counter calibration)")
    ap.add_argument("--cossim-only", type=int, default=0,
                    help="profiling helper: N eager UV-Prune similarity scores (72B hidden shape)")
    return ap.parse_args()


# ------------------------------------------------------------ byte counts --
def esize_of(w):
    return 4 if w.dtype == "f32" else 2


def verify_bytes(w, esize=None):
    """Algorithmic HBM bytes of one verify launch: K and V of the N + T visible
    rows, Q, O, mass and lse, each moved once."""
    esize = esize_of(w) if esize is None else esize
    N = int(w.lengths().sum()) + w.batch * w.T
    kv = 2 * N * w.hkv * w.head_dim * esize
    qo = 2 * w.batch * w.T * w.hq * w.head_dim * esize
    return kv + qo + 4 * w.batch * w.n_cap() + 4 * w.batch * w.hq * w.T


def gather_bytes(w, esize=None):
    esize = esize_of(w) if esize is None else esize
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


def cossim_bytes(w, esize=2):
    """Hidden states of layers 0 and L (the layer sum telescopes), score out."""
    m = int(w.m_per_seq().sum())
    return 2 * (m + w.batch * w.n_text) * w.hidden * esize + 4 * m


# ---------------------------------------------------------------- traffic --
def measured_traffic():
    """HBM bytes per verify launch from the committed rocprofv3 counter runs,
    or None when the kernel code changed since they were taken."""
    path = os.path.join(PROFILES, "verify_attn_llava72b_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    h = re.search(r"kernel code sha256: ([0-9a-f]{64})", text)
    t = re.search(r"traffic_bytes_per_launch: ([0-9.eE+]+)", text)
    if not h or not t:
        return None
    return float(t.group(1)) if kernel_code_digest() == h.group(1) else None


def kernel_code_digest():
    """sha256 of verify_attn.hip + common.h with comments and blank lines
    stripped: changes whenever the verify kernel's code does."""
    cur = hashlib.sha256()
    for f in VERIFY_SRCS:
        for line in open(f):
            code = re.sub(r"//.*", "", line).rstrip()
            if code:
                cur.update(code.encode() + b"\n")
    return cur.hexdigest()


# ------------------------------------------------------------ CPU baseline --
def cpu_model():
    """The first processor's identification in /proc/cpuinfo: the model name
    exactly as the host reports it (a virtual machine may give only the
    family name), with vendor, family, model, stepping and clock."""
    keys = ("model name", "vendor_id", "cpu family", "model", "stepping", "cpu MHz")
    found = {}
    try:
        for line in open("/proc/cpuinfo"):
            if not line.strip():
                break
            k, _, v = line.partition(":")
            k = k.strip()
            if k in keys and k not in found:
                found[k] = v.strip()
    except OSError:
        return "unknown"
    if not found:
        return "unknown"
    rest = ", ".join(f"{k} {found[k]}" for k in keys[1:] if k in found)
    return f"{found.get('model name', 'unknown')} ({rest})"


def oracle_single_layer_step(w, W, oracle, thread_limits):
    """Seconds the float64 oracle takes for one single-layer step of workload
    w on the host, once per entry of thread_limits (same inputs): verify of
    layer 1, the UV-Prune score over the masses of layers 0 and 1 (layer 0's
    mass exists before the step, as in the GPU step), top-k, the gather and
    accept."""
    import time as _t
    from threadpoolctl import threadpool_limits
    l0, l1 = W.make_verify_inputs(w, layer=0), W.make_verify_inputs(w, layer=1)
    f = lambda i: (W.storage_to_f64(i.q, i.dtype), W.storage_to_f64(i.k, i.dtype),
                   W.storage_to_f64(i.v, i.dtype))
    q0, k0, v0 = f(l0)
    mass0 = oracle.verify_attn(q0, k0, v0, l0.ctx_len, l0.scale)[2]
    q1, k1, v1 = f(l1)
    m = l1.m.astype(np.int32)
    K = w.keep_count(m).astype(np.int32)
    acc = W.make_accept_inputs(w)
    out = []
    for lim in thread_limits:
        with threadpool_limits(limits=lim):
            t0 = _t.perf_counter()
            mass1 = oracle.verify_attn(q1, k1, v1, l1.ctx_len, l1.scale)[2]
            mc = int(m.max())
            score = oracle.uvprune_score_mass(np.stack([mass0[:, :mc], mass1[:, :mc]]), m)
            idx = oracle.topk_select(score, m, K, max(1, int(K.max())))
            oracle.gather_kv(l1.k, l1.v, idx, K, m, np.full(w.batch, w.n_text),
                             max(1, int(K.max())) + w.n_text)
            oracle.spec_accept(acc.draft_logits, acc.target_logits, acc.draft_tokens, acc.u_accept,
                               acc.u_sample, acc.temperature)
            out.append(_t.perf_counter() - t0)
    return out


def cpu_baseline(w, layers_host, crit_layers, per_layer_ok):
    """Time the float64 oracle on host copies of the same inputs: a sample of
    the stacked step with every host core, and the single-layer steps of the
    tiny, 7B and 72B workloads with every core and with one thread."""
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
    singles = {}
    for name in ("tiny", "llava7b", "llava72b"):
        t_all, t_one = oracle_single_layer_step(W.WORKLOADS[name], W, oracle, (cores, 1))
        singles[name] = {"all_cores_ms": round(t_all * 1e3, 2), "one_thread_ms": round(t_one * 1e3, 2)}
    per_layer = np.mean(t_verify) + t_gather
    once = t_uv + t_topk + t_acc
    L = per_layer_ok
    us_per_layer = (per_layer + once / L) * 1e6
    cpu = cpu_model()
    return {
        "value": round(us_per_layer, 1), "unit": "us/layer", "cores": int(threads),
        "kind": "oracle",
        "sample": (f"float64 oracle on {len(layers_host)} of the {L} layers' verify inputs "
                   f"(mean {np.mean(t_verify):.2f} s/layer), gather of one layer "
                   f"({t_gather:.3f} s), UV-Prune over {crit_layers + 1} masses ({t_uv:.3f} s), "
                   f"top-k ({t_topk:.3f} s) and accept ({t_acc:.3f} s); per layer = verify + "
                   f"gather + (UV-Prune + top-k + accept) / {L}; BLAS threads {threads} of "
                   f"{cores} host cores in the process affinity; cpu {cpu}"),
        "cpu_model": cpu,
        "affinity_cores": cores,
        "single_layer_steps": singles,
        "single_layer_steps_note": ("the oracle's whole single-layer step (verify of one layer, "
                                    "UV-Prune, top-k, gather, accept) per workload, with every "
                                    "core and with one BLAS thread"),
    }


# ------------------------------------------------------------- the step --
class Step:
    """Inputs resident in HBM and the step's launches for one workload.

    Stacked: n_layers independent seeded layers (verify per layer; UV-Prune
    and top-k after layer L over the masses of layers 0..L; gather of every
    layer; accept).  Single layer: layer 0 (no salient boost) is the shallow
    reference whose mass exists before the step; the step verifies layer 1,
    scores, selects, gathers and accepts."""

    def __init__(self, torch, pv, W, w, stacked, dev):
        self.torch, self.pv, self.w, self.stacked = torch, pv, w, stacked
        NL = w.n_layers if stacked else 1
        L = w.crit_layers if stacked else 1
        self.NL, self.L = NL, L
        B, T, Hq, Hkv, D = w.batch, w.T, w.hq, w.hkv, w.head_dim
        n_cap = w.n_cap()
        lens = w.lengths()
        m_np = w.m_per_seq().astype(np.int32)
        K_np = w.keep_count(m_np).astype(np.int32)
        k_cap = max(1, int(K_np.max()))
        dst_cap = k_cap + w.n_text
        self.m_np, self.lens = m_np, lens
        tdt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
        self.Kc = torch.zeros((NL, B, Hkv, n_cap, D), dtype=tdt, device=dev)
        self.Vc = torch.zeros_like(self.Kc)
        self.Q = torch.zeros((NL, B, T, Hq, D), dtype=tdt, device=dev)
        for l in range(NL):
            layer_id = l if stacked else 1
            boost = W.crit_boost(w, layer_id) if stacked else 3.0
            W.make_verify_layer_torch(w, layer_id, boost, dev,
                                      k_out=self.Kc[l], v_out=self.Vc[l], q_out=self.Q[l])
        q0 = k0 = v0 = None
        if not stacked:
            q0, k0, v0 = W.make_verify_layer_torch(w, 1, 0.0, dev)
        self.ctx = torch.from_numpy(lens.astype(np.int32)).to(dev)
        self.m_t = torch.from_numpy(m_np).to(dev)
        self.k_t = torch.from_numpy(K_np).to(dev)
        self.tail_b = self.m_t.clone()
        self.tail_l = torch.full((B,), w.n_text, dtype=torch.int32, device=dev)
        acc = W.make_accept_inputs(w)
        self.temperature = acc.temperature
        self.dl = torch.from_numpy(acc.draft_logits).to(dev)
        self.tl = torch.from_numpy(acc.target_logits).to(dev)
        self.tok = torch.from_numpy(acc.draft_tokens).to(dev)
        self.ua = torch.from_numpy(acc.u_accept).to(dev)
        self.us = torch.from_numpy(acc.u_sample).to(dev)
        self.out = torch.empty((B, T, Hq, D), dtype=tdt, device=dev)
        self.lse = torch.empty((B, Hq, T), dtype=torch.float32, device=dev)
        self.crit = torch.zeros((L + 1, B, n_cap), dtype=torch.float32, device=dev)
        self.mass_x = torch.empty((B, n_cap), dtype=torch.float32, device=dev)
        self.score = torch.empty((B, n_cap), dtype=torch.float32, device=dev)
        self.k_cap, self.dst_cap = k_cap, dst_cap
        self.idx = torch.empty((B, k_cap), dtype=torch.int32, device=dev)
        self.kd = torch.zeros((NL, B, Hkv, dst_cap, D), dtype=tdt, device=dev)
        self.vd = torch.zeros_like(self.kd)
        self.na = torch.empty(B, dtype=torch.int32, device=dev)
        self.nt = torch.empty(B, dtype=torch.int32, device=dev)
        self.tie = torch.empty(B, dtype=torch.int32, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)
        self.ws_v = pv.Workspace(dev)
        self.ws_a = pv.Workspace(dev)
        self.max_ctx = int(lens.max())
        if not stacked:  # the shallow reference layer's mass exists before the step
            pv.verify_attn(q0, k0, v0, self.ctx, max_ctx=self.max_ctx, out=self.out,
                           mass=self.crit[0], lse=self.lse, ws=self.ws_v, status=self.status)
        torch.cuda.synchronize()

    def verify(self, l, mass=None):
        self.pv.verify_attn(self.Q[l], self.Kc[l], self.Vc[l], self.ctx, max_ctx=self.max_ctx,
                            out=self.out, mass=self.mass_x if mass is None else mass,
                            lse=self.lse, ws=self.ws_v, status=self.status)

    def prune(self):
        # UV-Prune's MASS variation and top-k in one launch
        self.pv.uvprune_topk_mass(self.crit, self.m_t, self.k_t, self.k_cap, score=self.score,
                                  idx=self.idx, status=self.status)

    def gather(self):
        self.pv.gather_kv(self.Kc, self.Vc, self.idx, self.k_t, self.tail_b, self.tail_l,
                          self.dst_cap, k_dst=self.kd, v_dst=self.vd, status=self.status)

    def accept(self):
        self.pv.spec_accept(self.dl, self.tl, self.tok, self.ua, self.us, self.temperature,
                            n_accepted=self.na, next_token=self.nt, near_tie=self.tie,
                            ws=self.ws_a, status=self.status)

    def step(self):
        for l in range(self.NL):
            if self.stacked:
                self.verify(l, self.crit[l] if l <= self.L else self.mass_x)
            else:
                self.verify(0, self.crit[1])
            if l == (self.L if self.stacked else 0):
                self.prune()
        self.gather()
        self.accept()

    def bytes(self):
        w = self.w
        return self.NL * (verify_bytes(w) + gather_bytes(w)) + uvprune_bytes(w) \
            + topk_bytes(w) + accept_bytes(w)


def capture(torch, fn):
    """A HIP graph of fn() (after one eager warm-up run on a side stream)."""
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        fn()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    torch.cuda.synchronize()
    return g


def time_replays(torch, run, n):
    """Mean ms per call of run() over n calls, HIP events on the current stream."""
    run()
    torch.cuda.synchronize()
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(n):
        run()
    b.record()
    torch.cuda.synchronize()
    return a.elapsed_time(b) / n


def replay_percentiles(torch, run, n, per_call=1):
    """(mean, p10, p50, p90) ms per call over n replays of run(), each
    bracketed by HIP events on the current stream (per_call calls each)."""
    run()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(n)]
    for a, b in ev:
        a.record()
        run()
        b.record()
    torch.cuda.synchronize()
    t = np.array([a.elapsed_time(b) for a, b in ev]) / per_call
    p10, p50, p90 = np.percentile(t, [10, 50, 90])
    return float(t.mean()), float(p10), float(p50), float(p90)


def copy_bandwidth(torch, dev, nbytes, reps):
    """Device-to-device copy GB/s (bytes read + written) for copies moving
    nbytes each.  The copies cycle over enough distinct buffers (>= 2 GiB in
    all) that no source is still in the 256 MB Infinity Cache when it is read
    again, as the verify launches cycle over the layers' caches."""
    n = max(1, -(-(2 << 30) // nbytes))
    bufs = [(torch.ones(nbytes // 4, dtype=torch.bfloat16, device=dev),
             torch.empty(nbytes // 4, dtype=torch.bfloat16, device=dev)) for _ in range(n)]

    def run():
        for s, d in bufs:
            d.copy_(s)

    g = capture(torch, run)
    ms = time_replays(torch, g.replay, reps) / n
    del bufs, g
    torch.cuda.empty_cache()
    return nbytes / (ms * 1e-3) / 1e9


def stage_times(torch, st, reps, pct=None):
    """Graph-timed mean us of each stage of the step (`reps` verify launches,
    cycling over the layers, or 10 launches of another stage per graph).
    With a dict `pct`, also each stage's [p10, p50, p90] over 10 replays."""
    out = {}
    g = capture(torch, lambda: [st.verify((7 * r + 3) % st.NL) for r in range(reps)])
    graphs = [("verify", g, reps)]
    for name, fn in (("uvprune+topk", st.prune), ("gather", st.gather), ("accept", st.accept)):
        graphs.append((name, capture(torch, lambda: [fn() for _ in range(10)]), 10))
    for name, g, k in graphs:
        if pct is None:
            out[name] = time_replays(torch, g.replay, 5) * 1e3 / k
        else:
            mean, p10, p50, p90 = replay_percentiles(torch, g.replay, 10, k)
            out[name] = mean * 1e3
            pct[name] = [round(p10 * 1e3, 2), round(p50 * 1e3, 2), round(p90 * 1e3, 2)]
    return out


def single_layer_record(torch, pv, W, name, dev, steps):
    w = W.WORKLOADS[name]
    st = Step(torch, pv, W, w, False, dev)
    g = capture(torch, st.step)
    ms, p10, p50, p90 = replay_percentiles(torch, g.replay, steps)
    pct = {}
    stg = stage_times(torch, st, 20, pct)
    vb = verify_bytes(w)
    rec = {
        "us_per_step": round(ms * 1e3, 2),
        "us_per_step_p10_p50_p90": [round(p10 * 1e3, 2), round(p50 * 1e3, 2), round(p90 * 1e3, 2)],
        "stages_us_p10_p50_p90": pct,
        "step_bytes": st.bytes(),
        "step_tbs": round(st.bytes() / (ms * 1e-3) / 1e12, 3),
        "stages_us": {k: round(v, 2) for k, v in stg.items()},
        "verify_tbs": round(vb / (stg["verify"] * 1e-6) / 1e12, 3),
        "verify_frac_of_peak": round(vb / (stg["verify"] * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
        "device_status": int(st.status.item()),
    }
    del st, g
    torch.cuda.empty_cache()
    return rec


def cossim_inputs(torch, w, dev):
    """Seeded hidden states of layers 0 and L (bf16) with the row counts."""
    B, m, n, Dh = w.batch, int(w.m_per_seq().max()), w.n_text, w.hidden
    gen = torch.Generator(device=dev)
    gen.manual_seed(260319610)
    hv = torch.randn((2, B, m, Dh), device=dev, generator=gen).to(torch.bfloat16)
    ht = torch.randn((2, B, n, Dh), device=dev, generator=gen).to(torch.bfloat16)
    m_t = torch.full((B,), m, dtype=torch.int32, device=dev)
    n_t = torch.full((B,), n, dtype=torch.int32, device=dev)
    return hv, ht, m_t, n_t


def cossim_record(torch, pv, W, dev):
    """UV-Prune similarity criterion on the 72B shape: layers 0 and L of the
    hidden states (the layer sum telescopes), bf16, hidden size 8192."""
    w = W.WORKLOADS["llava72b"]
    hv, ht, m_t, n_t = cossim_inputs(torch, w, dev)
    B, m = w.batch, hv.shape[2]
    score = torch.empty((B, m), dtype=torch.float32, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    ws = pv.Workspace(dev)

    def fn():
        pv.uvprune_score_cossim(hv, ht, m_t, n_t, score=score, ws=ws, status=status)

    g = capture(torch, fn)
    ms = time_replays(torch, g.replay, 20)
    nb = cossim_bytes(w)
    rec = {"workload": "llava72b hidden states, layers 0 and 20, D_h 8192, bf16",
           "us": round(ms * 1e3, 2), "bytes": nb,
           "tbs": round(nb / (ms * 1e-3) / 1e12, 3),
           "frac_of_peak": round(nb / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
           "device_status": int(status.item())}
    del hv, ht, g
    torch.cuda.empty_cache()
    return rec


def epilogue_record(torch, pv, W, dev):
    """A prefill layer's epilogue at the 72B hidden shape (12,544 visual and
    256 text rows, D_h 8192, bf16): the residual add with the layer's COSSIM
    criterion fused in (pvlm_prefill_epilogue_cossim), against the add
    followed by a separate criterion pass over the stored rows.  Bytes of the
    fused call: prev and delta read, the sum written, once each."""
    w = W.WORKLOADS["llava72b"]
    B, m, n, Dh = w.batch, int(w.m_per_seq().max()), w.n_text, w.hidden
    gen = torch.Generator(device=dev)
    gen.manual_seed(4242)
    bf = torch.bfloat16
    vp = torch.randn((B, m, Dh), device=dev, generator=gen).to(bf)
    vd = torch.randn((B, m, Dh), device=dev, generator=gen).to(bf)
    tp = torch.randn((B, n, Dh), device=dev, generator=gen).to(bf)
    td = torch.randn((B, n, Dh), device=dev, generator=gen).to(bf)
    vo, to = torch.empty_like(vp), torch.empty_like(tp)
    crit = torch.empty((B, m), dtype=torch.float32, device=dev)
    m_t = torch.full((B,), m, dtype=torch.int32, device=dev)
    n_t = torch.full((B,), n, dtype=torch.int32, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    ws = pv.Workspace(dev)

    def fused():
        pv.prefill_epilogue_cossim(vp, vd, tp, td, m_t, n_t, vis_out=vo, txt_out=to, crit=crit,
                                   ws=ws, status=status)

    def separate():
        torch.add(vp, vd, out=vo)
        torch.add(tp, td, out=to)
        pv.uvprune_criterion_cossim(vo, to, m_t, n_t, out=crit, ws=ws, status=status)

    res = {}
    for name, fn in (("fused", fused), ("separate", separate)):
        g = capture(torch, lambda: [fn() for _ in range(5)])
        res[name] = time_replays(torch, g.replay, 5) * 1e3 / 5
        del g
    nb = 3 * (m + n) * Dh * 2 * B
    rec = {"workload": "llava72b hidden states: 12544 visual + 256 text rows, D_h 8192, bf16",
           "fused_us": round(res["fused"], 2), "separate_us": round(res["separate"], 2),
           "fused_bytes": nb, "fused_tbs": round(nb / (res["fused"] * 1e-6) / 1e12, 3),
           "device_status": int(status.item())}
    del vp, vd, tp, td, vo, to
    torch.cuda.empty_cache()
    return rec


def rope_record(torch, pv, W, dev):
    """pvlm_rope_append at the 72B layer shape (T = 9 verify rows, 64 query and
    8 KV heads, D = 128, bf16, M-RoPE sections 16/24/24), 80 launches per
    graph replay.  Bytes: the rows read and written (q, k, v in; q, k, v out)."""
    w = W.WORKLOADS["llava72b"]
    B, T, Hq, Hkv, D = w.batch, w.T, w.hq, w.hkv, w.head_dim
    n_cap = w.n_cap()
    gen = torch.Generator(device=dev)
    gen.manual_seed(2603)
    q = torch.randn((B, T, Hq, D), device=dev, generator=gen).to(torch.bfloat16)
    kn = torch.randn((B, T, Hkv, D), device=dev, generator=gen).to(torch.bfloat16)
    vn = torch.randn((B, T, Hkv, D), device=dev, generator=gen).to(torch.bfloat16)
    kc = torch.zeros((B, Hkv, n_cap, D), dtype=torch.bfloat16, device=dev)
    vc = torch.zeros_like(kc)
    ctx = torch.from_numpy(w.lengths().astype(np.int32)).to(dev)
    p1 = ctx[:, None] + torch.arange(T, dtype=torch.int32, device=dev)[None, :]
    pos = torch.stack([p1, p1, p1]).contiguous()
    q_out = torch.empty_like(q)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    reps = 80

    def fn():
        for _ in range(reps):
            pv.rope_append(q, kn, vn, pos, ctx, kc, vc, base=w.rope_base, sections=(16, 24, 24),
                           q_out=q_out, status=status)

    g = capture(torch, fn)
    ms = time_replays(torch, g.replay, 10) / reps
    nb = 2 * B * T * (Hq + 2 * Hkv) * D * 2 + 4 * (3 * B * T + B)
    rec = {"workload": "llava72b verify rows: T 9, Hq 64, Hkv 8, D 128, bf16, M-RoPE 16/24/24",
           "us": round(ms * 1e3, 2), "bytes": nb, "bound": "latency",
           "device_status": int(status.item())}
    del q, kn, vn, kc, vc, g
    torch.cuda.empty_cache()
    return rec


def paged_record(torch, pv, W, dev, reps=20):
    """Verify attention on the batch-4 ragged layer (lengths in [16384, 33280],
    Hq 40, Hkv 8, D 128, bf16) from a padded cache and from paged pools of 32-
    and 256-row pages scattered over the pool; the same data and launch plan
    (max_ctx), graph-timed over `reps` launches each."""
    w = W.WORKLOADS["qwen32b"]
    q, k, v = W.make_verify_layer_torch(w, 1, 3.0, dev)
    lens = w.lengths()
    ctx = torch.from_numpy(lens.astype(np.int32)).to(dev)
    max_ctx = int(lens.max())
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    out = torch.empty_like(q)
    mass = torch.empty((w.batch, w.n_cap()), dtype=torch.float32, device=dev)
    lse = torch.empty((w.batch, w.hq, w.T), dtype=torch.float32, device=dev)
    ws = pv.Workspace(dev)

    def padded():
        pv.verify_attn(q, k, v, ctx, max_ctx=max_ctx, out=out, mass=mass, lse=lse, ws=ws,
                       status=status)

    g = capture(torch, lambda: [padded() for _ in range(reps)])
    us_pad = time_replays(torch, g.replay, 5) * 1e3 / reps
    del g
    ref = (out.clone(), mass.clone())
    vb = verify_bytes(w)
    rec = {"workload": "qwen32b verify, batch 4 ragged 16384..33280, Hq 40, Hkv 8, D 128, bf16",
           "bytes": vb, "padded_us": round(us_pad, 2),
           "padded_frac_of_peak": round(vb / (us_pad * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
           "paged": {}}
    for P in (32, 256):
        table, n_pages = W.page_table(lens + w.T, P, seed=P)
        kp, vp = W.to_pages(k, table, n_pages, P), W.to_pages(v, table, n_pages, P)
        tab = torch.from_numpy(table).to(dev)
        pmass = torch.empty((w.batch, table.shape[1] * P), dtype=torch.float32, device=dev)

        def paged():
            pv.verify_attn_paged(q, kp, vp, tab, ctx, max_ctx=max_ctx, out=out, mass=pmass,
                                 lse=lse, ws=ws, status=status)

        g = capture(torch, lambda: [paged() for _ in range(reps)])
        us = time_replays(torch, g.replay, 5) * 1e3 / reps
        n = ref[1].shape[1]
        same = bool(torch.equal(out, ref[0]) and torch.equal(pmass[:, :n], ref[1]))
        rec["paged"][str(P)] = {"us": round(us, 2), "pool_pages": n_pages,
                                "frac_of_peak": round(vb / (us * 1e-6) / 1e9 / HBM_PEAK_GBS, 4),
                                "bit_equal_to_padded": same}
        del g, kp, vp
    rec["device_status"] = int(status.item())
    del q, k, v, ws
    torch.cuda.empty_cache()
    return rec


def overlap_record(torch, pv, W, dev, gamma=5, reps=50):
    """Stage II concurrency at the 7B attention shape (28 query / 4 KV heads,
    D 128, bf16): the draft's gamma decode steps (rope-append + verify, T = 1)
    over the compact cache [V*, X] (627 kept visual + 160 text rows) on a
    32-CU stream, beside the target's round (rope-append + verify of T =
    gamma + 1 rows over the 6,432-row cache, then accept over V = 152064) on a
    224-CU stream.  Each side is one HIP graph; times are per round."""
    w = W.WORKLOADS["llava7b"]
    Hq, Hkv, D, T = w.hq, w.hkv, w.head_dim, gamma + 1
    n_prompt = int(w.lengths()[0])
    m = n_prompt - w.n_text
    n_c = int(w.keep_count(np.array([m]))[0]) + w.n_text
    gen = torch.Generator(device=dev)
    gen.manual_seed(5)
    bf = torch.bfloat16
    rnd = lambda *sh: torch.randn(sh, device=dev, generator=gen).to(bf)
    kt, vt = rnd(1, Hkv, n_prompt + 64, D), rnd(1, Hkv, n_prompt + 64, D)
    kd, vd = rnd(1, Hkv, n_c + 64, D), rnd(1, Hkv, n_c + 64, D)
    qt, knt, vnt = rnd(1, T, Hq, D), rnd(1, T, Hkv, D), rnd(1, T, Hkv, D)
    qd, knd, vnd = rnd(1, 1, Hq, D), rnd(1, 1, Hkv, D), rnd(1, 1, Hkv, D)
    ctx_t = torch.tensor([n_prompt], dtype=torch.int32, device=dev)
    pos_t = (n_prompt + torch.arange(T, dtype=torch.int32, device=dev))[None].contiguous()
    ctx_d = [torch.tensor([n_c + i], dtype=torch.int32, device=dev) for i in range(gamma)]
    pos_d = [torch.tensor([[n_prompt + i]], dtype=torch.int32, device=dev) for i in range(gamma)]
    V = w.vocab
    dl = torch.randn((1, gamma, V), device=dev, generator=gen)
    tl = torch.randn((1, gamma + 1, V), device=dev, generator=gen)
    tok = torch.randint(0, V, (1, gamma), device=dev, generator=gen).to(torch.int32)
    ua = torch.rand((1, gamma), device=dev, generator=gen, dtype=torch.float64)
    us = torch.rand((1,), device=dev, generator=gen, dtype=torch.float64)
    s_t, s_d = torch.cuda.Stream(), torch.cuda.Stream()
    pv.set_stream_cu_budget(s_t, 224)
    pv.set_stream_cu_budget(s_d, 32)
    ws_t, ws_d = pv.Workspace(dev), pv.Workspace(dev)
    st = torch.zeros(1, dtype=torch.int32, device=dev)

    def target_round():
        q = pv.rope_append(qt, knt, vnt, pos_t, ctx_t, kt, vt, base=w.rope_base, status=st)
        pv.verify_attn(q, kt, vt, ctx_t, want_lse=False, ws=ws_t, status=st)
        pv.spec_accept(dl, tl, tok, ua, us, 1.0, ws=ws_t, status=st)

    def draft_steps():
        for i in range(gamma):
            q = pv.rope_append(qd, knd, vnd, pos_d[i], ctx_d[i], kd, vd, base=w.rope_base, status=st)
            pv.verify_attn(q, kd, vd, ctx_d[i], want_mass=False, want_lse=False, ws=ws_d, status=st)

    graphs = {}
    for name, fn, s in (("target", target_round, s_t), ("draft", draft_steps, s_d)):
        with torch.cuda.stream(s):
            fn()                                  # sizes the workspaces, loads kernels
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            fn()
        torch.cuda.synchronize()
        graphs[name] = (g, s)

    def timed(names):
        for _ in range(3):
            for n in names:
                g, s = graphs[n]
                with torch.cuda.stream(s):
                    g.replay()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(reps):
            for n in names:
                g, s = graphs[n]
                with torch.cuda.stream(s):
                    g.replay()
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e6 / reps

    t_t = timed(["target"])
    t_d = timed(["draft"])
    t_both = timed(["target", "draft"])
    rec = {"workload": f"llava7b heads, gamma {gamma}: draft {gamma} x (rope + verify T=1) over "
                       f"{n_c} rows on 32 CUs beside target rope + verify T={T} over {n_prompt} rows "
                       f"+ accept (V {V}) on 224 CUs",
           "target_us": round(t_t, 2), "draft_us": round(t_d, 2), "both_us": round(t_both, 2),
           "overlap_frac": round((t_t + t_d - t_both) / min(t_t, t_d), 3),
           "timing": f"HIP graph per stream, {reps} rounds between host synchronisations",
           "device_status": int(st.item())}
    pv.set_stream_cu_budget(s_t, 0)
    pv.set_stream_cu_budget(s_d, 0)
    del graphs, ws_t, ws_d, kt, vt, kd, vd
    torch.cuda.empty_cache()
    return rec


def verify_plan(w, cus=256, xcds=8):
    """The verify launch plan the library picks for this shape: (row tiles per
    workgroup, row groups, splits, chunk tokens, resident, wide).  One
    workgroup per CU; rows split into groups of at most 5 tiles, more groups
    when the (batch, KV head) pairs are fewer than the XCDs; resident scores
    for chunks of at most 512 tokens; one group of 9 tiles (wide variant, two
    workgroups per CU) in place of two groups for streamed chunks."""
    rtt = -(-w.group * w.T // 16)
    n = int(w.lengths().max()) + w.T

    def layout(rg, slots=cus):
        per_launch = min(w.batch * w.hkv * rg, slots)
        splits = max(1, slots // per_launch)
        chunk = -(-(-(-n // splits)) // 32) * 32
        return per_launch, -(-n // chunk), chunk

    rg = -(-rtt // 5)
    if w.batch * w.hkv * rg < xcds and rtt > rg:
        rg = min(-(-xcds // (w.batch * w.hkv)), rtt)
    rt = -(-rtt // rg)
    per_launch, splits, chunk = layout(rg)
    resident = chunk <= 512
    wide = not resident and 5 < rtt <= 9 and w.batch * w.hkv >= xcds
    if wide:  # two workgroups per CU
        rg, rt = 1, 9
        per_launch, splits, chunk = layout(rg, 2 * cus)
    return rt, rg, per_launch, splits, chunk, resident, wide


def verify_kernel_label(w, cus=256, xcds=8):
    """The verify kernel variant of the launch plan (same-XCD exchange when
    every group's workgroups share an XCD)."""
    rt, rg, per_launch, splits, chunk, resident, wide = verify_plan(w, cus, xcds)
    grid = -(-per_launch * splits // 8) * 8
    local = grid % xcds == 0 and (grid // xcds) % splits == 0
    where = "same-XCD" if local else "cross-XCD"
    if wide:
        return f"verify_wide_kernel<{w.head_dim},{where}>"
    return f"verify_mfma_kernel<{w.head_dim},{rt},{'resident' if resident else 'stream'},{where}>"


def teardown(torch, pv, *objs):
    """Release graphs, tensors and the binding's default buffers and wait for
    the device before the interpreter exits, so that nothing the GPU runtime
    (or a profiler attached to it) tears down at process exit is still
    referenced by live Python objects."""
    for o in objs:
        del o
    import gc
    gc.collect()
    pv.release_workspaces()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()


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
        del src, dst
        teardown(torch, pv)
        return

    if args.cossim_only:  # the similarity criterion's kernels, eager, on the 72B hidden shape
        w = W.WORKLOADS["llava72b"]
        hv, ht, m_t, n_t = cossim_inputs(torch, w, dev)
        score = torch.empty((w.batch, hv.shape[2]), dtype=torch.float32, device=dev)
        status = torch.zeros(1, dtype=torch.int32, device=dev)
        ws = pv.Workspace(dev)
        for _ in range(args.cossim_only):
            pv.uvprune_score_cossim(hv, ht, m_t, n_t, score=score, ws=ws, status=status)
        torch.cuda.synchronize()
        print(json.dumps({"cossim_only": args.cossim_only, "bytes_per_call": cossim_bytes(w),
                          "status": int(status.item())}))
        del hv, ht, score, ws
        teardown(torch, pv)
        return

    w = W.WORKLOADS[args.workload]
    stacked = args.mode == "stacked"
    t0 = time.time()
    st = Step(torch, pv, W, w, stacked, dev)
    NL = st.NL
    log(f"inputs: {NL} layer(s), cache {2 * st.Kc.numel() * st.Kc.element_size() / 1e9:.2f} GB, "
        f"{time.time() - t0:.1f} s")

    if args.verify_only:
        # the launches as the bench times them: one graph of N verify
        # launches (one per layer, cycling), replayed once; captured without
        # an eager run, so the process makes no cooperative launch
        st.ws_v.get(pv.verify_attn_workspace_size(
            pv.PVLM_BF16 if w.dtype == "bf16" else pv.PVLM_F32, w.batch, w.T, w.hq, w.hkv,
            w.head_dim, w.n_cap(), st.max_ctx))
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=torch.cuda.Stream()):
            for r in range(args.verify_only):
                st.verify(r % NL)
        g.replay()
        torch.cuda.synchronize()
        print(json.dumps({"verify_only": args.verify_only, "status": int(st.status.item())}))
        del g, st
        teardown(torch, pv)
        return

    if args.gather_only:
        st.step()  # the kept indices of this step
        for _ in range(args.gather_only):
            st.gather()
        torch.cuda.synchronize()
        print(json.dumps({"gather_only": args.gather_only, "bytes_per_gather": NL * gather_bytes(w),
                          "status": int(st.status.item())}))
        del st
        teardown(torch, pv)
        return

    # eager warm-up (also sizes the workspaces before any capture)
    st.step()
    torch.cuda.synchronize()
    run = st.step
    graph_used = False
    if not args.no_graph:
        try:
            run = capture(torch, st.step).replay
            graph_used = True
        except Exception as e:  # capture unsupported: time eager launches
            log(f"graph capture failed ({type(e).__name__}: {e}); timing eager launches")
            torch.cuda.synchronize()
    for _ in range(args.warmup):
        run()
    torch.cuda.synchronize()
    st.status.zero_()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
    torch.cuda.synchronize()
    h0 = time.perf_counter()
    evs[0].record()
    for i in range(args.steps):
        run()
        evs[i + 1].record()
    torch.cuda.synchronize()
    host_s = time.perf_counter() - h0
    ms_step = evs[0].elapsed_time(evs[-1]) / args.steps
    per_step = np.array([evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps)])
    status = int(st.status.item())
    if status:
        log(f"device status {status} during the timed steps")

    # ---- per-stage times; verify is the dominant kernel: `reps` launches
    # (cycling over the layers) in one graph, events on the replaying stream
    # around whole replays give its mean launch duration, inter-kernel gaps
    # included.
    reps = args.kernel_reps
    vb = verify_bytes(w)
    stages = None
    if graph_used:
        stages = stage_times(torch, st, reps)
        k_mean = stages["verify"]
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
        st.verify((7 * r + 3) % NL)
        b.record()
    torch.cuda.synchronize()
    del blocker
    eager_us = float(np.mean([a.elapsed_time(b) * 1e3 for a, b in evs][2:]))
    if stages is None:
        k_mean = eager_us
    achieved = vb / (k_mean * 1e-6) / 1e9
    copy_same = copy_bandwidth(torch, dev, 4 * (vb // 4), 5)
    copy_big = copy_bandwidth(torch, dev, 2 << 30, 5)

    step_bytes = st.bytes()
    us_layer = ms_step * 1e3 / NL
    traffic = measured_traffic()

    cpu = None
    if not args.no_cpu_baseline:
        hosts = []
        # a bounded sample: every fourth layer of the stack (20 layers)
        sample = [0] if not stacked else list(range(0, NL, 4))
        for l in sample:
            li = min(l, NL - 1)
            hosts.append((W.storage_to_f64(st.Q[li].float().cpu().numpy(), "f32"),
                          st.Kc[li].float().cpu().double().numpy(),
                          st.Vc[li].float().cpu().double().numpy(), st.lens))
        t0 = time.time()
        cpu = cpu_baseline(w, hosts, st.L, NL)
        log(f"cpu baseline {time.time() - t0:.1f} s")
    m_max = int(st.m_np.max())
    L_used = st.L
    del st, run
    torch.cuda.empty_cache()

    others = None
    cossim = rope = paged = overlap = epi = None
    if not args.no_extra and graph_used:
        others = {}
        for name in OTHER_CONFIGS:
            t0 = time.time()
            others[name] = single_layer_record(torch, pv, W, name, dev, 20)
            log(f"{name} single layer: {others[name]['us_per_step']} us/step "
                f"({time.time() - t0:.1f} s)")
        cossim = cossim_record(torch, pv, W, dev)
        log(f"cossim: {cossim['us']} us")
        rope = rope_record(torch, pv, W, dev)
        log(f"rope_append: {rope['us']} us")
        epi = epilogue_record(torch, pv, W, dev)
        log(f"prefill epilogue: {epi}")
        paged = paged_record(torch, pv, W, dev)
        log(f"paged verify: padded {paged['padded_us']} us, paged {paged['paged']}")
        overlap = overlap_record(torch, pv, W, dev)
        log(f"stage II overlap: {overlap}")

    rec = {
        "metric": METRIC,
        "value": round(us_layer, 3),
        "unit": "us/layer",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "ms_per_step_p10_p50_p90": [round(float(x), 4) for x in np.percentile(per_step, [10, 50, 90])],
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": f"{w.name}-{'stacked-%dL' % NL if stacked else 'single-layer'}",
            "batch": w.batch, "query_heads": w.hq, "kv_heads": w.hkv, "head_dim": w.head_dim,
            "visual_tokens": m_max, "text_tokens": w.n_text, "gamma": w.gamma,
            "verify_rows": w.T, "keep": f"{w.keep_num}/{w.keep_den}", "uvprune_layers": L_used,
            "vocab": w.vocab, "layers": NL, "criterion": "attention mass",
            "hip_graph": graph_used,
        },
        "achieved_hbm_tbs": round(step_bytes / (ms_step * 1e-3) / 1e12, 3),
        "step_bytes": step_bytes,
        "host_ms_per_step": round(host_s * 1e3 / args.steps, 4),
        "stages_us": {k: round(v, 2) for k, v in stages.items()} if stages else None,
        "copy_gbs": {"same_bytes_as_verify": round(copy_same, 1), "2GiB": round(copy_big, 1)},
        "roofline": {
            "bound": "hbm", "kernel": verify_kernel_label(w),
            "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "bytes_per_launch": vb, "launch_us": round(k_mean, 3),
            "launch_timing": ("graph of %d launches, events around replays" % reps
                              if graph_used else "eager launches, events around each"),
            "eager_launch_us": round(eager_us, 3),
            "frac_of_copy_same_bytes": round(achieved / copy_same, 4),
        },
        "other_configs": others,
        "cossim": cossim,
        "rope_append": rope,
        "prefill_epilogue": epi,
        "paged_kv": paged,
        "stage2_overlap": overlap,
        "cpu_baseline": cpu,
        "device_status": status,
    }
    print(json.dumps(rec), flush=True)
    teardown(torch, pv)


if __name__ == "__main__":
    main()
