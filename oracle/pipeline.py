"""Oracle: the parallel decoding pipeline's scheduling (pre-verify and
post-verify modes, draft rollback), as plain Python.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Follows Suppl. "Parallel Pipeline Details", Alg. (speculative_decoding), its
worked example with gamma = 3, and Sec. 4.2, Stage I (result iii: a startup
window is already drafted when prefill ends) and Stage II (the draft drafts the
next window while the target verifies the previous one).

The scheduler decides, round by round, what the target verifies and what the
draft drafts; the caller runs the two models and reports what the target
accepted.  One round overlaps one target forward (c t) with gamma draft
forwards (gamma t), so it lasts max(gamma, c) t.

Readings where the paper is silent or loose:

* Startup.  Prefill ends with the draft's own first token d0 followed by a
  startup window d1..d_gamma drafted while the target was still prefilling.
  The initial pre-verify decides d0 from the target's prefill output, so it
  runs no forward and takes no time.
* Pre-verify round (pending empty): the draft drafts gamma tokens from the
  committed prefix; the target verifies the first of them.  Accepted: it is
  committed, the other gamma - 1 become the pending window and the mode
  switches to post-verify.  Rejected: the target's token is committed, every
  draft is dropped and the mode stays pre-verify.
* Post-verify round: the target verifies the whole pending window while the
  draft drafts gamma tokens after it.  All accepted: the window is committed,
  the new drafts become the pending window, the mode stays post-verify (the
  target's token after the window is not used: the draft has already gone
  past it).  First rejection at j: the first j tokens and the target's token
  are committed, everything after is dropped and the mode resets to
  pre-verify.
* Post-verify needs a pending window: with gamma = 1 an accepted pre-verify
  leaves none, and the next round is a pre-verify round again.
* Rollback: after a rejection the draft keeps the cache entries of the
  committed tokens before the target's token and resumes from that token;
  ``draft_keep`` is that many output tokens.
* The loop ends once at least ``max_len`` tokens are committed (the output
  may overrun by the tokens of the last round).
* Adaptive draft length: the longest run of committed draft tokens not
  interrupted by a token of the target.
"""
from __future__ import annotations

PRE, POST, DONE = "pre", "post", "done"


class Pipeline:
    """Scheduler state: committed output, pending window, mode, clock."""

    def __init__(self, gamma, c, max_len):
        self.gamma, self.c, self.max_len = gamma, c, max_len
        self.out = []          # committed output tokens
        self.pending = []      # drafted, not yet verified
        self.mode = PRE
        self.started = False
        self.clock = 0.0       # in units of t
        self.rounds = 0        # rounds that ran a target forward
        self.run = 0           # current run of committed draft tokens
        self.max_run = 0
        self.draft_keep = 0
        self.log = []

    def start(self, startup):
        """startup = [d0, d1, ..., d_gamma]: the draft's tokens from prefill."""
        assert not self.started and len(startup) == self.gamma + 1
        self.pending = list(startup)
        self.started = True

    def plan(self):
        """What the round about to run does: (mode, verify positions, draft
        positions, cost), positions counted in the output sequence."""
        if len(self.out) >= self.max_len:
            self.mode = DONE
            return {"mode": DONE}
        n = len(self.out)
        if self.rounds == 0 and len(self.log) == 0:
            # initial pre-verify of d0 against the target's prefill output
            return {"mode": PRE, "verify_begin": n, "verify_count": 1,
                    "draft_begin": n + len(self.pending), "draft_count": 0, "cost": 0.0}
        cost = max(float(self.gamma), float(self.c))
        if self.mode == PRE:
            return {"mode": PRE, "verify_begin": n, "verify_count": 1,
                    "draft_begin": n, "draft_count": self.gamma, "cost": cost}
        return {"mode": POST, "verify_begin": n, "verify_count": len(self.pending),
                "draft_begin": n + len(self.pending), "draft_count": self.gamma, "cost": cost}

    def _commit_draft(self, toks):
        self.out.extend(toks)
        self.run += len(toks)
        self.max_run = max(self.max_run, self.run)

    def _commit_target(self, tok):
        self.out.append(tok)
        self.run = 0

    def finish(self, drafted, n_accepted, resampled=None):
        """Apply the round's outcome.  drafted: the draft's new tokens;
        n_accepted: how many verified tokens the target accepted; resampled:
        the target's token at the first rejection."""
        p = self.plan()
        assert p["mode"] != DONE and len(drafted) == p["draft_count"]
        assert 0 <= n_accepted <= p["verify_count"]
        if p["draft_count"]:
            # the draft runs from the committed prefix in pre-verify mode
            if p["mode"] == PRE:
                self.pending = list(drafted)
            else:
                self.pending = self.pending + list(drafted)
        verified = self.pending[:p["verify_count"]]
        rest = self.pending[p["verify_count"]:]
        self._commit_draft(verified[:n_accepted])
        if n_accepted == p["verify_count"]:
            self.pending = rest
            self.mode = POST if rest else PRE
        else:
            self.draft_keep = len(self.out)
            self._commit_target(resampled)
            self.pending = []
            self.mode = PRE
        self.clock += p["cost"]
        if p["cost"] > 0:
            self.rounds += 1
        self.log.append(dict(p, accepted=n_accepted, committed=len(self.out),
                             next_mode=self.mode, draft_keep=self.draft_keep))
        if len(self.out) >= self.max_len:
            self.mode = DONE


def run_greedy(target_next, draft_next, prompt, gamma, c, max_len):
    """Drive the pipeline with two greedy models (functions from a token
    sequence to its next token); the target accepts a draft token iff it is
    its own next token, else emits its own (Sec. 2.2 at temperature 0)."""
    pl = Pipeline(gamma, c, max_len)
    seq = list(prompt)
    startup = []
    for _ in range(gamma + 1):
        startup.append(draft_next(seq + startup))
    pl.start(startup)
    while True:
        p = pl.plan()
        if p["mode"] == DONE:
            break
        base = list(prompt) + pl.out
        if p["mode"] == PRE and p["draft_count"]:
            spec = []
        else:
            spec = list(pl.pending)
        drafted = []
        for _ in range(p["draft_count"]):
            drafted.append(draft_next(base + spec + drafted))
        window = (drafted if p["mode"] == PRE and p["draft_count"] else spec)[:p["verify_count"]]
        acc, res = 0, None
        for tok in window:
            want = target_next(base + window[:acc])
            if tok != want:
                res = want
                break
            acc += 1
        pl.finish(drafted, acc, res)
    return pl


def autoregressive(target_next, prompt, n):
    """The target alone, one token per forward."""
    seq = list(prompt)
    for _ in range(n):
        seq.append(target_next(seq))
    return seq[len(prompt):]
