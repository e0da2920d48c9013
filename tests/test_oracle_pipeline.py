"""Pins for the parallel decoding pipeline oracle (not gpu).

Checked against the supplement's worked example with gamma = 3
(tests/golden/pipeline_trace.txt: output, mode switches, rollback points,
three target rounds in 9t, adaptive draft length 5); the lossless property of
speculative decoding (Sec. 2.2) -- with greedy models the committed output is
the target's own autoregressive sequence whatever the draft proposes; and the
ideal parallel-SD time of the supplement's theorem when every draft token is
accepted.
"""
import math

import pytest

from golden_io import pipeline_trace
from oracle import pipeline as PL
from oracle import window as W


def test_worked_example_gamma3():
    fx = pipeline_trace()
    pl = PL.Pipeline(gamma=3, c=3.0, max_len=len(fx["output"]))
    pl.start(fx["startup"])
    modes, keeps = [], []
    for drafted, acc, tok in fx["rounds"]:
        pl.finish(drafted, acc, tok)
        modes.append(pl.log[-1]["next_mode"])
        keeps.append(str(pl.draft_keep) if tok is not None else "-")
    assert pl.out == fx["output"]
    assert pl.mode == PL.DONE and pl.plan()["mode"] == PL.DONE
    assert modes == fx["modes"]
    assert keeps == fx["draft_keep"]
    assert pl.rounds == fx["target_rounds"]
    assert pl.clock == fx["elapsed"]
    assert pl.max_run == fx["max_draft_run"]
    # what each round asked of the two models
    shape = [(r["mode"], r["verify_begin"], r["verify_count"], r["draft_begin"], r["draft_count"])
             for r in pl.log]
    assert shape == [("pre", 0, 1, 4, 0), ("post", 1, 3, 4, 3), ("post", 4, 3, 7, 3),
                     ("pre", 6, 1, 6, 3)]


def _mix(seq, salt):
    h = 2166136261 ^ salt
    for t in seq[-4:]:
        h = ((h ^ (t + 1)) * 16777619) & 0xFFFFFFFF
    return h ^ (len(seq) * 2654435761 & 0xFFFFFFFF)


def _models(vocab, miss_every):
    def target_next(seq):
        return _mix(seq, 1) % vocab

    def draft_next(seq):
        t = target_next(seq)
        if miss_every and _mix(seq, 7) % miss_every == 0:
            return (t + 1) % vocab
        return t
    return target_next, draft_next


@pytest.mark.parametrize("gamma", [1, 2, 3, 5, 8])
@pytest.mark.parametrize("miss_every", [0, 2, 3, 5, 11])
def test_lossless_with_greedy_models(gamma, miss_every):
    target_next, draft_next = _models(50, miss_every)
    for c in (1.0, 2.5, 5.0):
        pl = PL.run_greedy(target_next, draft_next, [3, 1, 4], gamma, c, 60)
        assert len(pl.out) >= 60
        assert pl.out == PL.autoregressive(target_next, [3, 1, 4], len(pl.out))
        # every target round commits at least one token
        assert pl.rounds <= len(pl.out)


@pytest.mark.parametrize("gamma", [1, 2, 3, 5, 9])
@pytest.mark.parametrize("c", [1.0, 3.0, 5.36, 9.0])
def test_full_acceptance_meets_the_ideal_theorem(gamma, c):
    target_next, _ = _models(40, 0)
    n = 12
    pl = PL.run_greedy(target_next, target_next, [0], gamma, c, 1 + n * gamma)
    assert len(pl.out) == 1 + n * gamma
    assert pl.rounds == n and pl.max_run == len(pl.out)
    # after the free startup pre-verify, gamma tokens per round of max(gamma, c) t
    assert pl.clock / (len(pl.out) - 1) == pytest.approx(W.t_psd_ideal(c, gamma))


def test_draft_always_wrong_commits_one_target_token_per_round():
    target_next, _ = _models(40, 0)

    def draft_next(seq):
        return (target_next(seq) + 1) % 40
    pl = PL.run_greedy(target_next, draft_next, [5], 4, 4.0, 20)
    assert len(pl.out) == 20 and pl.max_run == 0
    assert pl.rounds == 19 and pl.clock == 19 * 4.0
    assert all(r["mode"] == "pre" and r["accepted"] == 0 for r in pl.log)
    assert [r["draft_keep"] for r in pl.log] == list(range(20))


def test_round_bookkeeping_invariants():
    target_next, draft_next = _models(30, 3)
    pl = PL.run_greedy(target_next, draft_next, [1, 2], 4, 4.0, 200)
    prev = 0
    for r in pl.log:
        rejected = r["accepted"] < r["verify_count"]
        assert r["committed"] - prev == r["accepted"] + (1 if rejected else 0)
        assert r["next_mode"] == ("pre" if rejected else "post")
        if rejected:
            assert r["draft_keep"] == r["committed"] - 1
        if r["mode"] == "post":
            assert r["verify_count"] in (3, 4)   # gamma - 1 after a pre-verify, else gamma
        prev = r["committed"]
    assert math.isclose(pl.clock, pl.rounds * 4.0)
