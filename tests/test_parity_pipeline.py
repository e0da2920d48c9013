"""Parity of the library's parallel decoding scheduler (pvlm_pd_*) with the
oracle.

The scheduler is host code (no device pointer, no stream), so these run
without a GPU.  Both are driven in lockstep with the same verdicts: the
supplement's gamma = 3 example, and greedy toy models (the target accepts a
draft token iff it is its own next token).  Every round's plan and the state
after it must match exactly, and the output must be the target's own
autoregressive sequence.
"""
import pytest

import paper_2603_19610_amd as P
from golden_io import pipeline_trace
from oracle import pipeline as PL

PLAN_KEYS = ("mode", "verify_begin", "verify_count", "draft_begin", "draft_count", "cost")


def _same_plan(lib_plan, ora_plan):
    if ora_plan["mode"] == "done":
        assert lib_plan["mode"] == "done"
        return
    assert {k: lib_plan[k] for k in PLAN_KEYS} == {k: ora_plan[k] for k in PLAN_KEYS}


def _same_state(s, pl):
    st = s.stats()
    assert s.output() == pl.out
    assert s.pending() == pl.pending
    assert st["mode"] == pl.plan()["mode"]
    assert st["target_rounds"] == pl.rounds
    assert st["max_draft_run"] == pl.max_run
    assert st["draft_keep"] == pl.draft_keep
    assert st["elapsed"] == pl.clock


def test_worked_example_gamma3():
    fx = pipeline_trace()
    vocab = {w: i for i, w in enumerate(sorted({w for r in fx["rounds"] for w in r[0]} |
                                               set(fx["startup"]) | set(fx["output"])))}
    words = {i: w for w, i in vocab.items()}
    s = P.Scheduler(3, 3.0, len(fx["output"]))
    pl = PL.Pipeline(3, 3.0, len(fx["output"]))
    s.start([vocab[w] for w in fx["startup"]])
    pl.start([vocab[w] for w in fx["startup"]])
    for drafted, acc, tok in fx["rounds"]:
        _same_plan(s.plan(), pl.plan())
        ids = [vocab[w] for w in drafted]
        t = None if tok is None else vocab[tok]
        s.finish(ids, acc, t)
        pl.finish(ids, acc, t)
        _same_state(s, pl)
    assert [words[i] for i in s.output()] == fx["output"]
    st = s.stats()
    assert st["mode"] == "done" and st["target_rounds"] == fx["target_rounds"]
    assert st["elapsed"] == fx["elapsed"] and st["max_draft_run"] == fx["max_draft_run"]
    s.close()


def _mix(seq, salt):
    h = 2166136261 ^ salt
    for t in seq[-4:]:
        h = ((h ^ (t + 1)) * 16777619) & 0xFFFFFFFF
    return h ^ (len(seq) * 2654435761 & 0xFFFFFFFF)


def _drive(gamma, c, max_len, miss_every, vocab=64, prompt=(2, 7, 1)):
    def target_next(seq):
        return _mix(seq, 3) % vocab

    def draft_next(seq):
        t = target_next(seq)
        return (t + 1) % vocab if miss_every and _mix(seq, 11) % miss_every == 0 else t

    s = P.Scheduler(gamma, c, max_len)
    pl = PL.Pipeline(gamma, c, max_len)
    startup = []
    for _ in range(gamma + 1):
        startup.append(draft_next(list(prompt) + startup))
    s.start(startup)
    pl.start(startup)
    while True:
        p = s.plan()
        _same_plan(p, pl.plan())
        if p["mode"] == "done":
            break
        base = list(prompt) + s.output()
        spec = [] if (p["mode"] == "pre" and p["draft_count"]) else s.pending()
        drafted = []
        for _ in range(p["draft_count"]):
            drafted.append(draft_next(base + spec + drafted))
        window = (drafted if not spec else spec)[:p["verify_count"]]
        acc, res = 0, None
        for tok in window:
            want = target_next(base + window[:acc])
            if tok != want:
                res = want
                break
            acc += 1
        s.finish(drafted, acc, res)
        pl.finish(drafted, acc, res)
        _same_state(s, pl)
    out = s.output()
    assert out == PL.autoregressive(target_next, list(prompt), len(out))
    s.close()
    return pl


@pytest.mark.parametrize("gamma", [1, 2, 3, 5, 9, 16])
@pytest.mark.parametrize("miss_every", [0, 2, 4, 7])
def test_lockstep_with_greedy_models(gamma, miss_every):
    for c in (1.0, 3.0, 5.36, 9.0):
        pl = _drive(gamma, c, 80, miss_every)
        assert len(pl.out) >= 80


def test_rejects_bad_use():
    with pytest.raises(P.PvlmError):
        P.Scheduler(0, 3.0, 10)
    with pytest.raises(P.PvlmError):
        P.Scheduler(3, 0.0, 10)
    with pytest.raises(P.PvlmError):
        P.Scheduler(3, float("inf"), 10)
    with pytest.raises(P.PvlmError):
        P.Scheduler(3, 3.0, 0)
    s = P.Scheduler(3, 3.0, 10)
    with pytest.raises(P.PvlmError):
        s.plan()                      # before start
    with pytest.raises(ValueError):
        s.start([1, 2, 3])            # needs gamma + 1 tokens
    s.start([1, 2, 3, 4])
    with pytest.raises(P.PvlmError):
        s.start([1, 2, 3, 4])         # twice
    with pytest.raises(P.PvlmError):
        s.finish([5], 1)              # startup round drafts nothing
    with pytest.raises(P.PvlmError):
        s.finish([], 2)               # verifies one token
    assert s.stats()["committed"] == 0 and s.pending() == [1, 2, 3, 4]
    s.finish([], 1)
    assert s.output() == [1] and s.pending() == [2, 3, 4]
    s.close()


def test_finish_after_done_and_short_buffers():
    import ctypes
    s = P.Scheduler(2, 2.0, 1)
    s.start([4, 5, 6])
    s.finish([], 1)
    assert s.plan()["mode"] == "done"
    with pytest.raises(P.PvlmError):
        s.finish([], 0)
    L = P.lib()
    n = ctypes.c_int(0)
    buf = (ctypes.c_int32 * 1)()
    assert L.pvlm_pd_pending(s._h, buf, 1, ctypes.byref(n)) == 2   # 2 pending, room for 1
    assert n.value == 2 and buf[0] == 5
    assert L.pvlm_pd_output(s._h, None, 1, ctypes.byref(n)) == 1
    assert L.pvlm_pd_output(s._h, None, 0, None) == 1
    assert L.pvlm_pd_plan(None, None) == 1
    s.close()
