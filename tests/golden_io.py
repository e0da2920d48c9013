"""Readers for the hand-computed fixtures in tests/golden/."""
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _lines(name):
    with open(os.path.join(GOLDEN, name)) as f:
        for raw in f:
            line = raw.split("#", 1)[0].strip()
            if line:
                yield line


def nums(tokens):
    return np.array([float(t) for t in tokens], dtype=np.float64)


def verify_cases():
    cases, cur = [], None
    for line in _lines("verify_attention.txt"):
        key, *rest = line.split()
        if key == "case":
            cur = {"name": rest[0]}
        elif key == "end":
            cases.append(cur)
            cur = None
        else:
            cur[key] = nums(rest)
    return cases


def similarity_fixture():
    out = {"cos": []}
    for line in _lines("uvprune_similarity.txt"):
        key, rest = line.split(None, 1)
        if key == "cos":
            a, b, e = [p.split() for p in rest.split("|")]
            out["cos"].append((nums(a), nums(b), float(e[0])))
        else:
            out[key] = nums(rest.split())
    return out


def topk_fixture():
    groups, cur = [], None
    for line in _lines("topk_select.txt"):
        key, rest = line.split(None, 1)
        if key == "scores":
            cur = {"scores": np.array([float(t) for t in rest.split()], dtype=np.float32),
                   "k": []}
            groups.append(cur)
        elif key == "k":
            kk, ids = rest.split("|")
            cur["k"].append((int(kk), [int(t) for t in ids.split()]))
    return groups


def accept_fixture(name="spec_accept.txt"):
    out = {"cases": []}
    for line in _lines(name):
        key, rest = line.split(None, 1)
        if key == "case":
            u, e = rest.split("|")
            ua, us = [float(t) for t in u.split()]
            na, nt = [int(t) for t in e.split()]
            out["cases"].append((ua, us, na, nt))
        else:
            out[key] = nums(rest.split())
    return out


def window_fixture():
    """The paper's printed speed ratios, integer windows and worked example."""
    out = {"ratio": [], "gamma": [], "example": []}
    for line in _lines("window_size.txt"):
        key, *rest = line.split()
        if key == "ratio" or key == "gamma":
            pair, alpha, t_p, t_q, val = rest
            out[key].append((pair, float(alpha), float(t_p), float(t_q), float(val)))
        elif key == "example":
            out["example"].append(tuple(float(v) for v in rest))
        elif key == "window_gain":
            out["window_gain"] = float(rest[0])
    return out


def pipeline_trace():
    """The gamma = 3 pipeline example: startup tokens, scripted rounds and
    the expected outcome."""
    out = {"rounds": []}
    for line in _lines("pipeline_trace.txt"):
        key, rest = line.split(None, 1)
        if key == "round":
            drafted, outcome = rest.split("|")
            drafted = [] if drafted.strip() == "-" else drafted.split()
            acc, tok = outcome.split()
            out["rounds"].append((drafted, int(acc), None if tok == "-" else tok))
        elif key in ("startup", "output", "modes", "draft_keep"):
            out[key] = rest.split()
        else:
            out[key] = float(rest)
    return out
