"""Helpers for the GPU parity tests: host arrays <-> device tensors and the
tolerances of the parity gates."""
import sys

import numpy as np
import torch

import workloads as W


def dev():
    return torch.device("cuda", 0)


def to_dev(a: np.ndarray, dtype: str = None):
    """numpy -> device tensor; uint16 arrays are bf16 bit patterns."""
    t = torch.from_numpy(np.ascontiguousarray(a))
    if a.dtype == np.uint16:
        t = t.view(torch.bfloat16)
    return t.to(dev())


def to_host_f64(t: torch.Tensor) -> np.ndarray:
    return t.detach().to(torch.float64).cpu().numpy()


def f64(a, dtype):
    return W.storage_to_f64(a, dtype)


def note(msg: str):
    """Name the case before each GPU step (flushed, so a crash still shows it)."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


# parity gates
OUT_ABS, OUT_REL = 2e-2, 2e-2      # attention output (bf16), abs + rel
LSE_ABS = 1e-4                     # log-sum-exp: fp32 softmax statistics
MASS_REL, MASS_FLOOR = 1e-4, 1e-9  # mass: rel + floor * Hq * T
SCORE_REL = 1e-4                   # pruning score


def assert_out(got, ref):
    err = np.abs(got - ref)
    lim = OUT_ABS + OUT_REL * np.abs(ref)
    bad = err > lim
    assert not bad.any(), f"out: {bad.sum()} of {bad.size} beyond tolerance, max err {err.max():.3g}"


def assert_lse(got, ref):
    err = np.abs(got - ref)
    assert err.max() <= LSE_ABS + 1e-6 * np.abs(ref).max(), f"lse max err {err.max():.3g}"


def assert_mass(got, ref, hq, T):
    err = np.abs(got - ref)
    lim = MASS_REL * np.abs(ref) + MASS_FLOOR * hq * T
    bad = err > lim
    assert not bad.any(), (f"mass: {bad.sum()} of {bad.size} beyond tolerance, "
                           f"max rel err {(err / np.maximum(np.abs(ref), 1e-30)).max():.3g}")
