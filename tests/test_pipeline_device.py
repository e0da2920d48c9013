"""GPU: the parallel decoding pipeline with both models on the device, on two
streams at once (Sec. 4.2, Stage II: the draft drafts the next window while
the target verifies the current one; Suppl. B, pre- and post-verify rounds
and draft rollback).

The two "models" are one-layer stand-ins at the 7B attention shape (28 query
heads, 4 KV heads, D = 128), built from this library's kernels: the new
tokens' query/key/value rows come from seeded embedding tables, are rotated
and appended by pvlm_rope_append, attend over the cache with pvlm_verify_attn,
and an output head (a seeded fp32 matrix) turns the attention output into
logits.  The target attends over the whole 6,432-row prompt cache.  The draft
attends over the compact cache [V*, X] that UV-Prune, top-k and pvlm_gather_kv
build from it (a tenth of the visual rows, by the target's attention mass)
and uses a perturbed output head, so it disagrees with the target now and
then.  The draft runs on its own stream with a 32-CU budget and the target
(verify + pvlm_spec_accept) on another with the remaining 224 CUs, so their
waiting kernels may overlap.  The draft rolls back by truncating its device
ctx_len to the longest prefix of its cache rows that is still valid.

At temperature 0 the committed output must be the target's own greedy
sequence (the lossless property of Sec. 2.2): target-only decoding, one token
per forward and teacher-forced on the committed prefix, must rank every
committed token first, up to the rounding of the bf16 attention output (the
pipeline computes the same logits inside verify windows of other lengths).
The scheduler must take the oracle's decisions given the kernel's verdicts.
"""
import numpy as np
import pytest
import torch

import paper_2603_19610_amd as pv
import workloads as W
from gpu_util import note
from oracle import pipeline as PL

pytestmark = pytest.mark.gpu

V = 512
Hq, Hkv, D = 28, 4, 128
BASE = 1.0e4
EMB_QK = 2.5


class Model:
    """Embeddings, output head and a KV cache; forward() runs on the current
    stream and never synchronises."""

    def __init__(self, emb, wo, k_cache, v_cache, dev):
        self.eq, self.ek, self.ev = emb
        self.wo = wo
        self.k, self.v = k_cache, v_cache
        self.ctx = torch.zeros(1, dtype=torch.int32, device=dev)
        self.ws = pv.Workspace(dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)

    def forward(self, toks, pos0, ctx):
        """toks: int64 device [T]; rows appended at cache rows ctx .. ctx+T-1
        with positions pos0 .. pos0+T-1 (int32 device scalars); returns
        logits [T][V] fp32."""
        T = toks.numel()
        ar = torch.arange(T, dtype=torch.int32, device=toks.device)
        pos = (pos0 + ar)[None].contiguous()
        self.ctx.copy_(ctx.view(1))
        q = self.eq[toks][None].contiguous()
        kn = self.ek[toks][None].contiguous()
        vn = self.ev[toks][None].contiguous()
        qr = pv.rope_append(q, kn, vn, pos, self.ctx, self.k, self.v, base=BASE, status=self.status)
        out, _, _ = pv.verify_attn(qr, self.k, self.v, self.ctx, want_mass=False, want_lse=False,
                                   ws=self.ws, status=self.status)
        self.last_out = out.float().reshape(T, Hq * D)
        return self.last_out @ self.wo.t()


def _setup(dev, seed, noise, cap_extra):
    w = W.WORKLOADS["llava7b"]
    n_prompt = int(w.lengths()[0])                  # 6272 visual + 160 text rows
    gen = torch.Generator(device=dev)
    gen.manual_seed(seed)
    # queries and keys of generated tokens scaled up, so a new token attends
    # mostly to the generated rows (which the two models share) and the draft
    # agrees with the target often enough to exercise post-verify rounds
    emb = tuple((sc * torch.randn((V, h, D), device=dev, generator=gen)).to(torch.bfloat16)
                for h, sc in ((Hq, EMB_QK), (Hkv, EMB_QK), (Hkv, 1.0)))
    wo = torch.randn((V, Hq * D), device=dev, generator=gen) / (Hq * D) ** 0.5
    wo_d = wo + noise * torch.randn((V, Hq * D), device=dev, generator=gen) / (Hq * D) ** 0.5
    q0, k0, v0 = W.make_verify_layer_torch(w, 1, 3.0, dev)
    n_cap = n_prompt + cap_extra
    kt = torch.zeros((1, Hkv, n_cap, D), dtype=torch.bfloat16, device=dev)
    vt = torch.zeros_like(kt)
    kt[:, :, :n_prompt] = k0[:, :, :n_prompt]
    vt[:, :, :n_prompt] = v0[:, :, :n_prompt]
    # UV-Prune over the target's attention mass of the prompt's verify rows
    # (one layer: criterion stack [0, mass]), top-k, gather into [V*, X]
    ctx = torch.tensor([n_prompt], dtype=torch.int32, device=dev)
    _, mass, _ = pv.verify_attn(q0, k0, v0, ctx)
    m = n_prompt - w.n_text
    stack = torch.zeros((2, 1, m), dtype=torch.float32, device=dev)
    stack[1] = mass[:, :m]
    score = pv.uvprune_score_mass(stack, torch.tensor([m], dtype=torch.int32, device=dev))
    keep = int(w.keep_count(np.array([m]))[0])
    idx = pv.topk_select(score, torch.tensor([m], dtype=torch.int32, device=dev),
                         torch.tensor([keep], dtype=torch.int32, device=dev), keep)
    n_c = keep + w.n_text
    kd, vd = pv.gather_kv(kt, vt, idx, torch.tensor([keep], dtype=torch.int32, device=dev),
                          torch.tensor([m], dtype=torch.int32, device=dev),
                          torch.tensor([w.n_text], dtype=torch.int32, device=dev),
                          n_c + cap_extra)
    torch.cuda.synchronize()
    target = Model(emb, wo, kt, vt, dev)
    draft = Model(emb, wo_d, kd, vd, dev)
    return target, draft, n_prompt, n_c


def _check_greedy(target, n_prompt, p_last, out, dev):
    """The committed tokens against target-only decoding, one token (T = 1)
    per forward, teacher-forced on the committed prefix (on copies of the
    cache).  Each committed token must be a greedy choice of the target's
    logits up to rounding: the pipeline computes those logits inside verify
    windows of other lengths, whose launch plans round the bf16 attention
    output differently.  A logit then moves by at most
    sum_j |dO_j| |wo[v, j]| with |dO_j| <= 2 ulp of bf16 (2^-7 |O_j|), so the
    committed token's logit must be within that bound, taken for both
    candidates, of the maximum.  Returns (positions where the committed token
    is not the exact argmax, the smallest top-2 gap)."""
    k, v = target.k.clone(), target.v.clone()
    ref = Model((target.eq, target.ek, target.ev), target.wo, k, v, dev)
    wabs = target.wo.abs()
    prev, off, gaps = p_last, 0, []
    for i, tok in enumerate(out):
        c = torch.tensor(n_prompt + i, dtype=torch.int32, device=dev)
        lg = ref.forward(torch.tensor([prev], device=dev), c, c)[0]
        o = ref.last_out.abs().reshape(-1)
        best = int(torch.argmax(lg))
        top = torch.topk(lg, 2).values
        gaps.append(float(top[0] - top[1]))
        if tok != best:
            bound = 2.0 ** -7 * float((wabs[best] @ o) + (wabs[tok] @ o))
            assert float(lg[best] - lg[tok]) <= bound, (i, tok, best, float(lg[best] - lg[tok]), bound)
            off += 1
        prev = tok
    assert int(ref.status.item()) == 0
    return off, min(gaps)


def _run(gamma, c, max_len, noise, seed):
    dev = torch.device("cuda", 0)
    target, draft, n_prompt, n_c = _setup(dev, seed, noise, max_len + 4 * gamma + 8)
    p_last = 7
    ref_k, ref_v = target.k.clone(), target.v.clone()  # the prompt cache, before the run appends
    s_t, s_d = torch.cuda.Stream(), torch.cuda.Stream()
    pv.set_stream_cu_budget(s_t, 224)
    pv.set_stream_cu_budget(s_d, 32)
    assert pv.stream_cu_budget(s_t) == 224 and pv.stream_cu_budget(s_d) == 32
    sched = pv.Scheduler(gamma, c, max_len)
    pl = PL.Pipeline(gamma, c, max_len)
    drow = []            # tokens whose rows follow the draft's compact prompt rows
    dl_of = {}           # generated-sequence index -> the draft's logits row for that token
    it = lambda x: torch.tensor(x, dtype=torch.int32, device=dev)

    def draft_after(xgen, count, first_event=None):
        """Enqueue on s_d: roll the draft cache back to its longest valid
        prefix of xgen[:-1], feed the rest of xgen, then draft `count`
        tokens.  Returns device tensors (tokens [count], logits [count][V]);
        the caller records the draft's rows (drow) once the tokens are known."""
        nonlocal drow
        lcp = 0
        while lcp < min(len(drow), len(xgen) - 1) and drow[lcp] == xgen[lcp]:
            lcp += 1
        drow = drow[:lcp]        # rollback: rows past lcp are rewritten below
        toks = torch.empty(count, dtype=torch.int64, device=dev)
        logits = torch.empty((count, V), dtype=torch.float32, device=dev)
        with torch.cuda.stream(s_d):
            feed = torch.tensor(xgen[lcp:], dtype=torch.int64, device=dev)
            lg = draft.forward(feed, it(n_prompt + lcp), it(n_c + lcp))[-1]
            L = len(xgen)       # drafted token i is fed at generated index L + i
            for i in range(count):
                logits[i] = lg
                toks[i] = torch.argmax(lg)
                if i == 0 and first_event is not None:
                    first_event.record(s_d)
                if i + 1 < count:
                    lg = draft.forward(toks[i:i + 1], it(n_prompt + L + i), it(n_c + L + i))[-1]
        return toks, logits

    # startup: d0 .. d_gamma drafted while the target prefills
    toks, logits = draft_after([p_last], gamma + 1)
    torch.cuda.synchronize()
    startup = [int(x) for x in toks.cpu()]
    drow = [p_last] + startup[:-1]
    for i, tok in enumerate(startup):
        dl_of[1 + i] = logits[i]
    sched.start(startup)
    pl.start(startup)
    zeros = torch.zeros(64, dtype=torch.float64, device=dev)
    rounds = rejected = full = 0
    while True:
        p = sched.plan()
        if p["mode"] == "done":
            break
        out = sched.output()
        sgen = [p_last] + out
        pre_draft = p["mode"] == "pre" and p["draft_count"] > 0
        spec = [] if pre_draft else sched.pending()
        ev = torch.cuda.Event() if pre_draft else None
        if p["draft_count"]:
            d_toks, d_logits = draft_after(sgen + spec, p["draft_count"], ev)
        # target: verify [last committed token] + window
        with torch.cuda.stream(s_t):
            if pre_draft:
                s_t.wait_event(ev)
                window = d_toks[:1]
                wl = d_logits[:1]
            else:
                wtoks = spec[:p["verify_count"]]
                window = torch.tensor(wtoks, dtype=torch.int64, device=dev)
                wl = torch.stack([dl_of[len(sgen) + i] for i in range(len(wtoks))])
            g = window.numel()
            feed = torch.cat([torch.tensor([sgen[-1]], dtype=torch.int64, device=dev), window])
            c0 = n_prompt + len(sgen) - 1
            tl = target.forward(feed, it(c0), it(c0))
            n, y, _ = pv.spec_accept(wl[None].contiguous(), tl[None].contiguous(),
                                     window.to(torch.int32)[None].contiguous(),
                                     zeros[:g].view(1, g), zeros[:1], 0.0, ws=target.ws,
                                     status=target.status)
            n_h, y_h = n.cpu(), y.cpu()
        torch.cuda.synchronize()
        drafted = [int(x) for x in d_toks.cpu()] if p["draft_count"] else []
        if p["draft_count"]:
            base_len = len(sgen + spec)
            drow = sgen + spec + drafted[:-1]
            for i in range(len(drafted)):
                dl_of[base_len + i] = d_logits[i]
        acc = int(n_h[0])
        tok = None if acc == g else int(y_h[0])
        rejected += tok is not None
        full += acc == g
        rounds += 1
        sched.finish(drafted, acc, tok)
        pl.finish(drafted, acc, tok)
        assert sched.output() == pl.out and sched.pending() == pl.pending
    out = sched.output()
    assert int(target.status.item()) == 0 and int(draft.status.item()) == 0
    target.k.copy_(ref_k)
    target.v.copy_(ref_v)
    off, gap = _check_greedy(target, n_prompt, p_last, out, dev)
    note(f"pipeline on device gamma={gamma} c={c} noise={noise}: {len(out)} tokens, "
         f"{off} within rounding of a tie, min top-2 gap {gap:.3g}")
    assert rejected > 0 and full > 0
    st = sched.stats()
    assert st["target_rounds"] == pl.rounds and st["elapsed"] == pl.clock
    pv.set_stream_cu_budget(s_t, 0)
    pv.set_stream_cu_budget(s_d, 0)
    sched.close()
    return rounds, rejected, full


@pytest.mark.parametrize("gamma,c,noise,seed", [(3, 3.0, 0.5, 5), (5, 5.0, 0.3, 6)])
def test_pipeline_both_models_on_two_streams(gamma, c, noise, seed):
    rounds, rejected, full = _run(gamma, c, 40, noise, seed)
    note(f"  {rounds} rounds, {rejected} ending in a rejection, {full} fully accepted")


def test_budget_rejects_bad_values():
    s = torch.cuda.Stream()
    for bad in (7, 12, 300, -8):
        with pytest.raises(pv.PvlmError):
            pv.set_stream_cu_budget(s, bad)
    pv.set_stream_cu_budget(s, 256)        # the whole device: no budget
    assert pv.stream_cu_budget(s) == 0
    pv.set_stream_cu_budget(s, 64)
    assert pv.stream_cu_budget(s) == 64
    pv.set_stream_cu_budget(s, 0)
    assert pv.stream_cu_budget(s) == 0
