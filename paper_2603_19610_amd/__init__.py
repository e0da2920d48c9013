"""Python binding of libpvlm.so, the MI355X (gfx950) ParallelVLM hot path.

Argument marshalling only: every step runs in the library's HIP kernels.
Tensors must be CUDA (HIP) tensors on the current device, C-contiguous, with
the dtypes the C ABI (include/pvlm.h) names.  Calls are enqueued on
``torch.cuda.current_stream()`` and return without synchronising.

There is no CPU fallback: if libpvlm.so is missing the import of a call's
library raises, telling the caller to build it.
"""
from __future__ import annotations

import ctypes
import os
import threading
from typing import Optional

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libpvlm.so")

PVLM_F32, PVLM_BF16 = 0, 1
PVLM_CRIT_MASS, PVLM_CRIT_COSSIM = 0, 1
PVLM_DEV_RANGE, PVLM_DEV_TIMEOUT, PVLM_DEV_PLACEMENT = 1, 2, 4

EXPORTS = (
    "pvlm_status_string", "pvlm_last_hip_error", "pvlm_version",
    "pvlm_set_stream_cu_budget", "pvlm_stream_cu_budget",
    "pvlm_verify_attn_workspace_size", "pvlm_verify_attn", "pvlm_verify_attn_paged",
    "pvlm_verify_attn_noalloc", "pvlm_verify_attn_noalloc_max_bytes",
    "pvlm_uvprune_workspace_size", "pvlm_uvprune_score", "pvlm_uvprune_criterion_cossim",
    "pvlm_prefill_epilogue_cossim",
    "pvlm_topk_workspace_size", "pvlm_topk_select", "pvlm_uvprune_topk_mass",
    "pvlm_gather_kv", "pvlm_gather_kv_paged",
    "pvlm_spec_accept_workspace_size", "pvlm_spec_accept",
    "pvlm_rope_append", "pvlm_rope_append_paged",
    "pvlm_speedup", "pvlm_window_size",
    "pvlm_pd_create", "pvlm_pd_destroy", "pvlm_pd_start", "pvlm_pd_plan", "pvlm_pd_finish",
    "pvlm_pd_output", "pvlm_pd_pending", "pvlm_pd_get_stats",
)


class PvlmError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str = ""):
        self.status = status
        msg = f"{where}: pvlm status {status}"
        if detail:
            msg += f" ({detail})"
        super().__init__(msg)


_lib = None
_lib_lock = threading.Lock()

_c = ctypes
_P = _c.c_void_p
_I = _c.c_int
_I64 = _c.c_int64
_SZ = _c.c_size_t
_F = _c.c_float
_D = _c.c_double

PVLM_ROUND_DOWN, PVLM_ROUND_UP, PVLM_ROUND_NEAREST, PVLM_ROUND_BEST = 0, 1, 2, 3
_ROUNDING = {"down": PVLM_ROUND_DOWN, "up": PVLM_ROUND_UP, "nearest": PVLM_ROUND_NEAREST,
             "best": PVLM_ROUND_BEST}


class SpeedupModel(_c.Structure):
    """pvlm_speedup_model: per-token times (units of the draft forward t) and
    speedups against target-only decoding."""
    _fields_ = [(n, _c.c_double) for n in (
        "t_sd_ideal", "t_psd_ideal", "t_sd", "t_psd", "t_psd_rollback",
        "v_sd_ideal", "v_psd_ideal", "v_sd", "v_psd", "v_psd_rollback",
        "expected_accepted", "expected_total")]

    def as_dict(self):
        return {n: getattr(self, n) for n, _ in self._fields_}


PVLM_PD_PRE_VERIFY, PVLM_PD_POST_VERIFY, PVLM_PD_DONE = 0, 1, 2
_PD_MODES = {PVLM_PD_PRE_VERIFY: "pre", PVLM_PD_POST_VERIFY: "post", PVLM_PD_DONE: "done"}


class PdRound(_c.Structure):
    """pvlm_pd_round: what one round of the parallel decoding pipeline runs."""
    _fields_ = [("mode", _c.c_int32), ("verify_begin", _c.c_int32),
                ("verify_count", _c.c_int32), ("draft_begin", _c.c_int32),
                ("draft_count", _c.c_int32), ("cost", _c.c_double)]


class PdStats(_c.Structure):
    """pvlm_pd_stats: the scheduler's counters."""
    _fields_ = [("mode", _c.c_int32), ("committed", _c.c_int32), ("pending", _c.c_int32),
                ("target_rounds", _c.c_int32), ("max_draft_run", _c.c_int32),
                ("draft_keep", _c.c_int32), ("elapsed", _c.c_double)]

_SIGS = {
    "pvlm_status_string": (_c.c_char_p, [_I]),
    "pvlm_last_hip_error": (_c.c_char_p, []),
    "pvlm_version": (_I, []),
    "pvlm_set_stream_cu_budget": (_I, [_P, _I]),
    "pvlm_stream_cu_budget": (_I, [_P]),
    "pvlm_verify_attn_workspace_size": (_SZ, [_I, _I, _I, _I, _I, _I, _I64, _I64]),
    "pvlm_verify_attn": (_I, [_I, _I, _I, _I, _I, _I, _I64, _I64, _F, _P, _P, _P, _P, _P, _P, _P,
                              _P, _SZ, _P, _P]),
    "pvlm_verify_attn_paged": (_I, [_I, _I, _I, _I, _I, _I, _I, _I, _I64, _I64, _F, _P, _P, _P,
                                    _P, _P, _P, _P, _P, _P, _SZ, _P, _P]),
    "pvlm_verify_attn_noalloc": (_I, [_I, _I, _I, _I, _I, _I, _I64, _I64, _F, _P, _P, _P, _P, _P,
                                      _P, _P, _P, _P]),
    "pvlm_verify_attn_noalloc_max_bytes": (_SZ, []),
    "pvlm_uvprune_workspace_size": (_SZ, [_I, _I, _I, _I64]),
    "pvlm_uvprune_score": (_I, [_I, _I, _I, _I64, _P, _P, _I, _I, _I64, _P, _P, _P, _P, _P, _SZ,
                                _P, _P]),
    "pvlm_uvprune_criterion_cossim": (_I, [_I, _I64, _P, _I, _I, _I64, _P, _P, _P, _P, _P, _SZ,
                                           _P, _P]),
    "pvlm_prefill_epilogue_cossim": (_I, [_I, _I64, _P, _I64, _P, _I, _I, _P, _P, _P, _P, _P, _P,
                                          _P, _P, _SZ, _P, _P]),
    "pvlm_topk_workspace_size": (_SZ, [_I, _I64]),
    "pvlm_topk_select": (_I, [_I, _I64, _P, _P, _I, _P, _P, _P, _SZ, _P, _P]),
    "pvlm_uvprune_topk_mass": (_I, [_I, _I, _I64, _P, _P, _P, _I, _P, _P, _P, _SZ, _P, _P]),
    "pvlm_gather_kv": (_I, [_I, _I, _I, _I, _I, _I64, _P, _P, _P, _P, _I, _P, _P, _I64, _P, _P,
                            _P, _P]),
    "pvlm_gather_kv_paged": (_I, [_I, _I, _I, _I, _I, _I, _I, _I64, _P, _P, _P, _P, _P, _I, _P,
                                  _P, _I64, _P, _P, _P, _P]),
    "pvlm_spec_accept_workspace_size": (_SZ, [_I, _I, _I]),
    "pvlm_spec_accept": (_I, [_I, _I, _I, _F, _P, _P, _P, _P, _P, _P, _P, _P, _P, _SZ, _P, _P]),
    "pvlm_speedup": (_I, [_D, _D, _I, _c.POINTER(SpeedupModel)]),
    "pvlm_window_size": (_I, [_D, _D, _I, _D, _I, _c.POINTER(_I), _c.POINTER(_D)]),
    "pvlm_rope_append": (_I, [_I, _I, _I, _I, _I, _I, _I64, _D, _P, _P, _P, _P, _P, _P, _P, _P,
                              _P, _P, _P]),
    "pvlm_rope_append_paged": (_I, [_I, _I, _I, _I, _I, _I, _I, _I, _I64, _D, _P, _P, _P, _P, _P,
                                    _P, _P, _P, _P, _P, _P, _P]),
    "pvlm_pd_create": (_I, [_I, _D, _I, _c.POINTER(_P)]),
    "pvlm_pd_destroy": (None, [_P]),
    "pvlm_pd_start": (_I, [_P, _P]),
    "pvlm_pd_plan": (_I, [_P, _c.POINTER(PdRound)]),
    "pvlm_pd_finish": (_I, [_P, _P, _I, _I, _c.c_int32]),
    "pvlm_pd_output": (_I, [_P, _P, _I, _c.POINTER(_I)]),
    "pvlm_pd_pending": (_I, [_P, _P, _I, _c.POINTER(_I)]),
    "pvlm_pd_get_stats": (_I, [_P, _c.POINTER(PdStats)]),
}


def lib():
    """The loaded libpvlm.so (loads it on first use; raises if not built)."""
    global _lib
    if _lib is None:
        with _lib_lock:
            if _lib is None:
                if not os.path.exists(LIB_PATH):
                    raise RuntimeError(
                        f"{LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; "
                        "g.build()'` or `python -m paper_2603_19610_amd.build`")
                L = ctypes.CDLL(LIB_PATH)
                for name, (res, args) in _SIGS.items():
                    fn = getattr(L, name)
                    fn.restype = res
                    fn.argtypes = args
                _lib = L
    return _lib


def _check(status: int, where: str):
    if status != 0:
        L = lib()
        detail = L.pvlm_status_string(status).decode()
        if status == 5:
            detail += ": " + L.pvlm_last_hip_error().decode()
        raise PvlmError(status, where, detail)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _need(t: torch.Tensor, name: str, dtype=None, device=None):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return t


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.bfloat16:
        return PVLM_BF16
    if t.dtype == torch.float32:
        return PVLM_F32
    raise ValueError(f"unsupported dtype {t.dtype}")


class Workspace:
    """A zero-initialised device scratch buffer that grows on demand.

    The library leaves its synchronisation words consistent after every call,
    so one buffer can serve successive calls on one stream (not concurrent
    calls: give each stream its own workspace).  A buffer that is outgrown is
    kept alive, not freed: a graph captured earlier, or a call still running,
    may use it.
    """

    def __init__(self, device=None):
        self.device = torch.device("cuda", torch.cuda.current_device()) if device is None else device
        self.buf = torch.zeros(256, dtype=torch.uint8, device=self.device)
        self._retired = []

    def get(self, nbytes: int) -> torch.Tensor:
        if nbytes > self.buf.numel():
            self._retired.append(self.buf)
            self.buf = torch.zeros(max(nbytes, 2 * self.buf.numel()), dtype=torch.uint8,
                                   device=self.device)
        return self.buf


# Default workspaces, one per (call kind, device, stream): calls on different
# streams never share counters or data.
_ws_cache = {}
# Default status words, one per device (see synchronize()).
_status_cache = {}


def _no_capture(what: str):
    if torch.cuda.is_current_stream_capturing():
        raise PvlmError(4, "status", f"cannot {what} during graph capture: call "
                        "default_status() once before capturing, or pass status=")


def _default_ws(kind: str) -> Workspace:
    key = (kind, torch.cuda.current_device(), torch.cuda.current_stream().cuda_stream)
    ws = _ws_cache.get(key)
    if ws is None:
        # (under graph capture the buffer comes from the graph's pool and its
        # zero fill replays with the graph, which leaves the counters consistent)
        ws = _ws_cache[key] = Workspace()
    return ws


def _status(status):
    """The caller's status word, or this device's default one."""
    if status is not None:
        return status
    dev = torch.cuda.current_device()
    st = _status_cache.get(dev)
    if st is None:
        _no_capture("allocate the default status word")
        st = _status_cache[dev] = torch.zeros(1, dtype=torch.int32, device=torch.device("cuda", dev))
    return st


def default_status() -> torch.Tensor:
    """The status word calls without an explicit ``status`` OR their device
    flags (PVLM_DEV_*) into, on the current device."""
    return _status(None)


def synchronize(raise_on_status: bool = True) -> int:
    """Wait for the current device, then read and clear its default status
    word.  Raises PvlmError when a call flagged a device-side condition (an
    out-of-range device size, a wait that gave up, a misplaced workgroup)
    unless ``raise_on_status`` is False; returns the flags."""
    torch.cuda.synchronize()
    st = _status(None)
    flags = int(st.item())
    if flags:
        st.zero_()
        torch.cuda.synchronize()
        if raise_on_status:
            raise PvlmError(flags, "device status", _flag_text(flags))
    return flags


def _flag_text(flags: int) -> str:
    names = [(PVLM_DEV_RANGE, "device size out of range"), (PVLM_DEV_TIMEOUT, "wait gave up"),
             (PVLM_DEV_PLACEMENT, "workgroup placement")]
    return ", ".join(n for bit, n in names if flags & bit)


def release_workspaces():
    """Drop the default workspaces and status words (every call using them must
    have completed, and no live graph may reference them)."""
    torch.cuda.synchronize()
    _ws_cache.clear()
    _status_cache.clear()


# ------------------------------------------------------------------ calls --
def set_stream_cu_budget(stream, cus: int):
    """Give ``stream`` (a torch.cuda.Stream) a compute-unit budget: its verify,
    long-row top-k and accept calls then plan for at most ``cus`` workgroups
    and launch as ordinary launches, so they may run beside calls on streams
    whose budgets sum with it to at most the device's compute units.  0
    removes the budget."""
    _check(lib().pvlm_set_stream_cu_budget(_P(stream.cuda_stream), int(cus)),
           "pvlm_set_stream_cu_budget")


def stream_cu_budget(stream) -> int:
    return int(lib().pvlm_stream_cu_budget(_P(stream.cuda_stream)))


def verify_attn_workspace_size(dtype: int, B, T, Hq, Hkv, D, n_cap, max_ctx) -> int:
    return int(lib().pvlm_verify_attn_workspace_size(dtype, B, T, Hq, Hkv, D, n_cap, max_ctx))


def verify_attn(q, k_cache, v_cache, ctx_len, *, scale: Optional[float] = None,
                max_ctx: Optional[int] = None, out=None, mass=None, lse=None,
                want_mass: bool = True, want_lse: bool = True, ws: Optional[Workspace] = None,
                status=None):
    """Verify attention + attention mass.  q [B][T][Hq][D]; caches [B][Hkv][n_cap][D];
    ctx_len [B] int32.  Returns (out, mass or None, lse or None)."""
    _need(q, "q")
    dev = q.device
    _need(k_cache, "k_cache", q.dtype, dev)
    _need(v_cache, "v_cache", q.dtype, dev)
    _need(ctx_len, "ctx_len", torch.int32, dev)
    B, T, Hq, D = q.shape
    Bk, Hkv, n_cap, Dk = k_cache.shape
    if Bk != B or Dk != D or tuple(v_cache.shape) != tuple(k_cache.shape) or ctx_len.numel() != B:
        raise ValueError("inconsistent verify_attn shapes")
    dt = _dt(q)
    if scale is None:
        scale = D ** -0.5
    if max_ctx is None:
        max_ctx = n_cap - T
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", q.dtype, dev)
    if mass is None and want_mass:
        mass = torch.empty((B, n_cap), dtype=torch.float32, device=dev)
    if mass is not None:
        _need(mass, "mass", torch.float32, dev)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, T), dtype=torch.float32, device=dev)
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
    need = verify_attn_workspace_size(dt, B, T, Hq, Hkv, D, n_cap, max_ctx)
    wsb = (ws or _default_ws("verify")).get(need)
    st = lib().pvlm_verify_attn(dt, B, T, Hq, Hkv, D, n_cap, max_ctx, float(scale), _ptr(q),
                                _ptr(k_cache), _ptr(v_cache), _ptr(ctx_len), _ptr(out), _ptr(mass),
                                _ptr(lse), _ptr(wsb), wsb.numel(), _ptr(_status(status)), _stream())
    _check(st, "pvlm_verify_attn")
    return out, mass, lse


def _pool_shape(k_pool, v_pool, page_table, dev, dtype, stacked=False):
    _need(k_pool, "k_pool", dtype, dev)
    _need(v_pool, "v_pool", dtype, dev)
    _need(page_table, "page_table", torch.int32, dev)
    want = 5 if stacked else 4
    if k_pool.dim() != want or tuple(v_pool.shape) != tuple(k_pool.shape):
        raise ValueError("pools must be [n_pages][Hkv][page][D]" if not stacked else
                         "pools must be [n_pages][Hkv][page][D] or [L][n_pages][Hkv][page][D]")
    if page_table.dim() != 2:
        raise ValueError("page_table must be [B][max_pages]")
    return tuple(k_pool.shape)


def verify_attn_paged(q, k_pool, v_pool, page_table, ctx_len, *, scale: Optional[float] = None,
                      max_ctx: Optional[int] = None, out=None, mass=None, lse=None,
                      want_mass: bool = True, want_lse: bool = True,
                      ws: Optional[Workspace] = None, status=None):
    """pvlm_verify_attn_paged: verify attention + mass over a paged cache.
    q [B][T][Hq][D] bf16; pools [n_pages][Hkv][page][D]; page_table
    [B][max_pages] int32; mass is [B][max_pages * page] by logical row."""
    _need(q, "q", torch.bfloat16)
    dev = q.device
    n_pages, Hkv, page, Dk = _pool_shape(k_pool, v_pool, page_table, dev, q.dtype)
    _need(ctx_len, "ctx_len", torch.int32, dev)
    B, T, Hq, D = q.shape
    if Dk != D or page_table.shape[0] != B or ctx_len.numel() != B:
        raise ValueError("inconsistent verify_attn_paged shapes")
    max_pages = page_table.shape[1]
    n_cap = max_pages * page
    if scale is None:
        scale = D ** -0.5
    if max_ctx is None:
        max_ctx = n_cap - T
    if out is None:
        out = torch.empty_like(q)
    _need(out, "out", q.dtype, dev)
    if mass is None and want_mass:
        mass = torch.empty((B, n_cap), dtype=torch.float32, device=dev)
    if mass is not None:
        _need(mass, "mass", torch.float32, dev)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, T), dtype=torch.float32, device=dev)
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
    need = verify_attn_workspace_size(PVLM_BF16, B, T, Hq, Hkv, D, n_cap, max_ctx)
    wsb = (ws or _default_ws("verify")).get(need)
    st = lib().pvlm_verify_attn_paged(PVLM_BF16, B, T, Hq, Hkv, D, page, max_pages, n_pages,
                                      max_ctx, float(scale), _ptr(q), _ptr(k_pool), _ptr(v_pool),
                                      _ptr(page_table), _ptr(ctx_len), _ptr(out), _ptr(mass),
                                      _ptr(lse), _ptr(wsb), wsb.numel(), _ptr(_status(status)),
                                      _stream())
    _check(st, "pvlm_verify_attn_paged")
    return out, mass, lse


def verify_attn_noalloc(q, k_cache, v_cache, ctx_len, *, out, mass=None, lse=None,
                        scale: Optional[float] = None, max_ctx: Optional[int] = None, status=None):
    """pvlm_verify_attn_noalloc: verify attention + mass with the library's
    fixed device scratch (no workspace, nothing allocated: ``out`` and the
    optional ``mass`` / ``lse`` are the caller's).  Calls that overlap on one
    GPU race on the shared scratch."""
    _need(q, "q")
    dev = q.device
    _need(k_cache, "k_cache", q.dtype, dev)
    _need(v_cache, "v_cache", q.dtype, dev)
    _need(ctx_len, "ctx_len", torch.int32, dev)
    _need(out, "out", q.dtype, dev)
    B, T, Hq, D = q.shape
    Bk, Hkv, n_cap, Dk = k_cache.shape
    if Bk != B or Dk != D or tuple(v_cache.shape) != tuple(k_cache.shape) or ctx_len.numel() != B:
        raise ValueError("inconsistent verify_attn shapes")
    if mass is not None:
        _need(mass, "mass", torch.float32, dev)
    if lse is not None:
        _need(lse, "lse", torch.float32, dev)
    st = lib().pvlm_verify_attn_noalloc(_dt(q), B, T, Hq, Hkv, D, n_cap,
                                        n_cap - T if max_ctx is None else max_ctx,
                                        float(D ** -0.5 if scale is None else scale), _ptr(q),
                                        _ptr(k_cache), _ptr(v_cache), _ptr(ctx_len), _ptr(out),
                                        _ptr(mass), _ptr(lse), _ptr(status), _stream())
    _check(st, "pvlm_verify_attn_noalloc")
    return out, mass, lse


def uvprune_score_mass(crit_stack, m, *, score=None, status=None):
    """score = UV-Prune variation over a criterion stack crit_stack [L+1][B][m_cap] fp32."""
    _need(crit_stack, "crit_stack", torch.float32)
    dev = crit_stack.device
    _need(m, "m", torch.int32, dev)
    Lp1, B, m_cap = crit_stack.shape
    if score is None:
        score = torch.empty((B, m_cap), dtype=torch.float32, device=dev)
    _need(score, "score", torch.float32, dev)
    st = lib().pvlm_uvprune_score(PVLM_CRIT_MASS, B, Lp1 - 1, m_cap, _ptr(m), _ptr(crit_stack),
                                  PVLM_F32, 0, 0, None, None, None, _ptr(score), None, 0,
                                  _ptr(_status(status)), _stream())
    _check(st, "pvlm_uvprune_score")
    return score


def uvprune_score_cossim(hs_vis, hs_txt, m, n_txt, *, score=None, ws=None, status=None):
    """Eq. (average_similarity) from hidden states hs_vis [L+1][B][m_cap][Dh], hs_txt [L+1][B][n_cap][Dh]."""
    _need(hs_vis, "hs_vis")
    dev = hs_vis.device
    _need(hs_txt, "hs_txt", hs_vis.dtype, dev)
    _need(m, "m", torch.int32, dev)
    _need(n_txt, "n_txt", torch.int32, dev)
    Lp1, B, m_cap, Dh = hs_vis.shape
    n_cap = hs_txt.shape[2]
    if hs_txt.shape[0] != Lp1 or hs_txt.shape[1] != B or hs_txt.shape[3] != Dh:
        raise ValueError("inconsistent hidden-state shapes")
    if score is None:
        score = torch.empty((B, m_cap), dtype=torch.float32, device=dev)
    _need(score, "score", torch.float32, dev)
    need = int(lib().pvlm_uvprune_workspace_size(PVLM_CRIT_COSSIM, B, Dh, n_cap))
    wsb = (ws or _default_ws("uvprune")).get(need)
    st = lib().pvlm_uvprune_score(PVLM_CRIT_COSSIM, B, Lp1 - 1, m_cap, _ptr(m), None,
                                  _dt(hs_vis), Dh, n_cap, _ptr(n_txt), _ptr(hs_vis), _ptr(hs_txt),
                                  _ptr(score), _ptr(wsb), wsb.numel(), _ptr(_status(status)), _stream())
    _check(st, "pvlm_uvprune_score")
    return score


def uvprune_criterion_cossim(hv, ht, m, n_txt, *, out=None, ws=None, status=None):
    """One layer: c[b,i] = sum_j cos(hv[b,i], ht[b,j]); hv [B][m_cap][Dh], ht [B][n_cap][Dh]."""
    _need(hv, "hv")
    dev = hv.device
    _need(ht, "ht", hv.dtype, dev)
    _need(m, "m", torch.int32, dev)
    _need(n_txt, "n_txt", torch.int32, dev)
    B, m_cap, Dh = hv.shape
    n_cap = ht.shape[1]
    if out is None:
        out = torch.empty((B, m_cap), dtype=torch.float32, device=dev)
    _need(out, "out", torch.float32, dev)
    need = int(lib().pvlm_uvprune_workspace_size(PVLM_CRIT_COSSIM, B, Dh, n_cap))
    wsb = (ws or _default_ws("uvprune")).get(need)
    st = lib().pvlm_uvprune_criterion_cossim(B, m_cap, _ptr(m), _dt(hv), Dh, n_cap, _ptr(n_txt),
                                             _ptr(hv), _ptr(ht), _ptr(out), _ptr(wsb), wsb.numel(),
                                             _ptr(_status(status)), _stream())
    _check(st, "pvlm_uvprune_criterion_cossim")
    return out


def prefill_epilogue_cossim(vis_prev, vis_delta, txt_prev, txt_delta, m, n_txt, *, vis_out=None,
                            txt_out=None, crit=None, ws=None, status=None):
    """pvlm_prefill_epilogue_cossim: the residual add of a prefill layer's
    visual [B][m_cap][Dh] and text [B][n_cap][Dh] rows with the layer's
    COSSIM criterion of the result fused in.  Outputs default to new tensors
    (pass vis_out=vis_prev for an in-place add).  Returns (vis_out, txt_out,
    crit [B][m_cap])."""
    _need(vis_prev, "vis_prev")
    dev = vis_prev.device
    dtp = vis_prev.dtype
    for t, name in ((vis_delta, "vis_delta"), (txt_prev, "txt_prev"), (txt_delta, "txt_delta")):
        _need(t, name, dtp, dev)
    _need(m, "m", torch.int32, dev)
    _need(n_txt, "n_txt", torch.int32, dev)
    B, m_cap, Dh = vis_prev.shape
    n_cap = txt_prev.shape[1]
    if (tuple(vis_delta.shape) != (B, m_cap, Dh) or tuple(txt_prev.shape) != (B, n_cap, Dh)
            or tuple(txt_delta.shape) != (B, n_cap, Dh)):
        raise ValueError("inconsistent prefill_epilogue_cossim shapes")
    if vis_out is None:
        vis_out = torch.empty_like(vis_prev)
    if txt_out is None:
        txt_out = torch.empty_like(txt_prev)
    _need(vis_out, "vis_out", dtp, dev)
    _need(txt_out, "txt_out", dtp, dev)
    if crit is None:
        crit = torch.empty((B, m_cap), dtype=torch.float32, device=dev)
    _need(crit, "crit", torch.float32, dev)
    need = int(lib().pvlm_uvprune_workspace_size(PVLM_CRIT_COSSIM, B, Dh, n_cap))
    wsb = (ws or _default_ws("uvprune")).get(need)
    st = lib().pvlm_prefill_epilogue_cossim(B, m_cap, _ptr(m), n_cap, _ptr(n_txt), _dt(vis_prev), Dh,
                                            _ptr(vis_prev), _ptr(vis_delta), _ptr(vis_out),
                                            _ptr(txt_prev), _ptr(txt_delta), _ptr(txt_out),
                                            _ptr(crit), _ptr(wsb), wsb.numel(), _ptr(_status(status)),
                                            _stream())
    _check(st, "pvlm_prefill_epilogue_cossim")
    return vis_out, txt_out, crit


def topk_select(score, m, k, k_cap: int, *, idx=None, ws=None, status=None):
    """Ascending kept indices [B][k_cap] (-1 padded)."""
    _need(score, "score", torch.float32)
    dev = score.device
    _need(m, "m", torch.int32, dev)
    _need(k, "k", torch.int32, dev)
    B, m_cap = score.shape
    if idx is None:
        idx = torch.empty((B, k_cap), dtype=torch.int32, device=dev)
    _need(idx, "idx", torch.int32, dev)
    need = int(lib().pvlm_topk_workspace_size(B, m_cap))
    wsb = (ws or _default_ws("topk")).get(need) if need else None
    st = lib().pvlm_topk_select(B, m_cap, _ptr(m), _ptr(k), int(k_cap), _ptr(score), _ptr(idx),
                                _ptr(wsb), 0 if wsb is None else wsb.numel(), _ptr(_status(status)),
                                _stream())
    _check(st, "pvlm_topk_select")
    return idx


def uvprune_topk_mass(crit_stack, m, k, k_cap: int, *, score=None, want_score: bool = True,
                      idx=None, ws=None, status=None):
    """pvlm_uvprune_topk_mass: the MASS score crit_stack[L] - crit_stack[0]
    ([L+1][B][m_cap] fp32) and its top-k in one launch.  Returns (score or
    None, idx)."""
    _need(crit_stack, "crit_stack", torch.float32)
    dev = crit_stack.device
    _need(m, "m", torch.int32, dev)
    _need(k, "k", torch.int32, dev)
    L1, B, m_cap = crit_stack.shape
    if score is None and want_score:
        score = torch.empty((B, m_cap), dtype=torch.float32, device=dev)
    if score is not None:
        _need(score, "score", torch.float32, dev)
    if idx is None:
        idx = torch.empty((B, k_cap), dtype=torch.int32, device=dev)
    _need(idx, "idx", torch.int32, dev)
    need = int(lib().pvlm_topk_workspace_size(B, m_cap))
    wsb = (ws or _default_ws("topk")).get(need) if need else None
    st = lib().pvlm_uvprune_topk_mass(B, L1 - 1, m_cap, _ptr(m), _ptr(crit_stack), _ptr(k),
                                      int(k_cap), _ptr(score), _ptr(idx), _ptr(wsb),
                                      0 if wsb is None else wsb.numel(), _ptr(_status(status)),
                                      _stream())
    _check(st, "pvlm_uvprune_topk_mass")
    return score, idx


def gather_kv(k_cache, v_cache, idx, k, tail_begin, tail_len, dst_cap: int, *, k_dst=None,
              v_dst=None, status=None):
    """Compact cache: kept rows then tail rows.  Caches are [B][Hkv][n_cap][D]
    (one layer) or [L][B][Hkv][n_cap][D] (a stacked cache, one launch);
    outputs have the same leading dims with dst_cap rows."""
    _need(k_cache, "k_cache")
    dev = k_cache.device
    _need(v_cache, "v_cache", k_cache.dtype, dev)
    _need(idx, "idx", torch.int32, dev)
    for name, t in (("k", k), ("tail_begin", tail_begin), ("tail_len", tail_len)):
        _need(t, name, torch.int32, dev)
    if k_cache.dim() == 4:
        n_layers, (B, Hkv, n_cap, D) = 1, k_cache.shape
    elif k_cache.dim() == 5:
        n_layers, B, Hkv, n_cap, D = k_cache.shape
    else:
        raise ValueError("k_cache must be [B][Hkv][n_cap][D] or [L][B][Hkv][n_cap][D]")
    if tuple(v_cache.shape) != tuple(k_cache.shape) or idx.shape[0] != B:
        raise ValueError("inconsistent gather_kv shapes")
    dst_shape = tuple(k_cache.shape[:-2]) + (dst_cap, D)
    if k_dst is None:
        k_dst = torch.zeros(dst_shape, dtype=k_cache.dtype, device=dev)
    if v_dst is None:
        v_dst = torch.zeros(dst_shape, dtype=k_cache.dtype, device=dev)
    _need(k_dst, "k_dst", k_cache.dtype, dev)
    _need(v_dst, "v_dst", k_cache.dtype, dev)
    if tuple(k_dst.shape) != dst_shape or tuple(v_dst.shape) != dst_shape:
        raise ValueError("destination shape mismatch")
    st = lib().pvlm_gather_kv(_dt(k_cache), n_layers, B, Hkv, D, n_cap, _ptr(k_cache),
                              _ptr(v_cache), _ptr(idx), _ptr(k), idx.shape[1], _ptr(tail_begin),
                              _ptr(tail_len), dst_cap, _ptr(k_dst), _ptr(v_dst),
                              _ptr(_status(status)), _stream())
    _check(st, "pvlm_gather_kv")
    return k_dst, v_dst


def gather_kv_paged(k_pool, v_pool, page_table, idx, k, tail_begin, tail_len, dst_cap: int, *,
                    k_dst=None, v_dst=None, status=None):
    """pvlm_gather_kv_paged: compact cache from a paged pool.  Pools are
    [n_pages][Hkv][page][D] (one layer) or [L][n_pages][Hkv][page][D]; one
    page_table [B][max_pages] serves every layer; outputs [(L,) B, Hkv, dst_cap, D]."""
    _need(k_pool, "k_pool")
    dev = k_pool.device
    if k_pool.dim() == 4:
        n_layers, (n_pages, Hkv, page, D) = 1, k_pool.shape
    elif k_pool.dim() == 5:
        n_layers, n_pages, Hkv, page, D = k_pool.shape
    else:
        raise ValueError("pools must be [n_pages][Hkv][page][D] or [L][n_pages][Hkv][page][D]")
    _need(v_pool, "v_pool", k_pool.dtype, dev)
    _need(page_table, "page_table", torch.int32, dev)
    _need(idx, "idx", torch.int32, dev)
    for name, t in (("k", k), ("tail_begin", tail_begin), ("tail_len", tail_len)):
        _need(t, name, torch.int32, dev)
    if tuple(v_pool.shape) != tuple(k_pool.shape) or page_table.dim() != 2:
        raise ValueError("inconsistent gather_kv_paged shapes")
    B, max_pages = page_table.shape
    if idx.shape[0] != B:
        raise ValueError("idx must be [B][k_cap]")
    dst_shape = ((n_layers,) if k_pool.dim() == 5 else ()) + (B, Hkv, dst_cap, D)
    if k_dst is None:
        k_dst = torch.zeros(dst_shape, dtype=k_pool.dtype, device=dev)
    if v_dst is None:
        v_dst = torch.zeros(dst_shape, dtype=k_pool.dtype, device=dev)
    _need(k_dst, "k_dst", k_pool.dtype, dev)
    _need(v_dst, "v_dst", k_pool.dtype, dev)
    if tuple(k_dst.shape) != dst_shape or tuple(v_dst.shape) != dst_shape:
        raise ValueError("destination shape mismatch")
    st = lib().pvlm_gather_kv_paged(_dt(k_pool), n_layers, B, Hkv, D, page, max_pages, n_pages,
                                    _ptr(k_pool), _ptr(v_pool), _ptr(page_table), _ptr(idx),
                                    _ptr(k), idx.shape[1], _ptr(tail_begin), _ptr(tail_len),
                                    dst_cap, _ptr(k_dst), _ptr(v_dst), _ptr(_status(status)),
                                    _stream())
    _check(st, "pvlm_gather_kv_paged")
    return k_dst, v_dst


def spec_accept(draft_logits, target_logits, draft_tokens, u_accept, u_sample,
                temperature: float, *, n_accepted=None, next_token=None, near_tie=None,
                ws: Optional[Workspace] = None, status=None):
    """Returns (n_accepted [B], next_token [B], near_tie [B]) int32 tensors."""
    _need(draft_logits, "draft_logits", torch.float32)
    dev = draft_logits.device
    _need(target_logits, "target_logits", torch.float32, dev)
    _need(draft_tokens, "draft_tokens", torch.int32, dev)
    _need(u_accept, "u_accept", torch.float64, dev)
    _need(u_sample, "u_sample", torch.float64, dev)
    B, gamma, V = draft_logits.shape
    if tuple(target_logits.shape) != (B, gamma + 1, V):
        raise ValueError("target_logits must be [B][gamma+1][V]")
    if n_accepted is None:
        n_accepted = torch.empty(B, dtype=torch.int32, device=dev)
    if next_token is None:
        next_token = torch.empty(B, dtype=torch.int32, device=dev)
    if near_tie is None:
        near_tie = torch.empty(B, dtype=torch.int32, device=dev)
    need = int(lib().pvlm_spec_accept_workspace_size(B, gamma, V))
    wsb = (ws or _default_ws("accept")).get(need)
    st = lib().pvlm_spec_accept(B, gamma, V, float(temperature), _ptr(draft_logits),
                                _ptr(target_logits), _ptr(draft_tokens), _ptr(u_accept),
                                _ptr(u_sample), _ptr(n_accepted), _ptr(next_token), _ptr(near_tie),
                                _ptr(wsb), wsb.numel(), _ptr(_status(status)), _stream())
    _check(st, "pvlm_spec_accept")
    return n_accepted, next_token, near_tie


__all__ = [
    "LIB_PATH", "EXPORTS", "PvlmError", "Workspace", "lib", "synchronize", "default_status",
    "release_workspaces", "set_stream_cu_budget", "stream_cu_budget",
    "verify_attn", "verify_attn_paged", "verify_attn_noalloc",
    "gather_kv_paged", "rope_append", "rope_append_paged",
    "verify_attn_workspace_size", "uvprune_score_mass", "uvprune_score_cossim",
    "uvprune_criterion_cossim", "prefill_epilogue_cossim", "topk_select", "uvprune_topk_mass", "gather_kv", "spec_accept",
    "PVLM_F32", "PVLM_BF16", "PVLM_CRIT_MASS", "PVLM_CRIT_COSSIM", "PVLM_DEV_RANGE",
    "PVLM_DEV_TIMEOUT", "PVLM_DEV_PLACEMENT",
]


def speedup(c: float, tau: float, gamma: int) -> dict:
    """pvlm_speedup: the speedup analysis for speed ratio c, acceptance rate
    tau and window gamma (host arithmetic, no GPU)."""
    out = SpeedupModel()
    _check(lib().pvlm_speedup(float(c), float(tau), int(gamma), _c.byref(out)), "speedup")
    return out.as_dict()


def window_size(t_p: float, t_q: float, rounding: str = "down", tau: float = 0.0,
                gamma_max: int = 64):
    """pvlm_window_size: the draft window gamma = T_p / T_q rounded as asked;
    returns (gamma, c)."""
    if rounding not in _ROUNDING:
        raise ValueError(f"rounding must be one of {sorted(_ROUNDING)}")
    g, c = _I(0), _D(0.0)
    _check(lib().pvlm_window_size(float(t_p), float(t_q), _ROUNDING[rounding], float(tau),
                                  int(gamma_max), _c.byref(g), _c.byref(c)), "window_size")
    return g.value, c.value


class Scheduler:
    """The library's parallel decoding scheduler (pvlm_pd_*): host state only.

    ``plan()`` says what the next round runs, ``finish()`` reports the
    target's verdict; tokens are Python ints."""

    def __init__(self, gamma: int, c: float, max_len: int):
        h = _P()
        _check(lib().pvlm_pd_create(int(gamma), float(c), int(max_len), _c.byref(h)),
               "pd_create")
        self._h = h
        self.gamma = int(gamma)

    def close(self):
        if self._h is not None and self._h.value:
            lib().pvlm_pd_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @staticmethod
    def _arr(tokens):
        tokens = list(tokens)
        return (_c.c_int32 * max(len(tokens), 1))(*tokens), len(tokens)

    def start(self, startup):
        arr, n = self._arr(startup)
        if n != self.gamma + 1:
            raise ValueError(f"startup needs gamma + 1 = {self.gamma + 1} tokens")
        _check(lib().pvlm_pd_start(self._h, arr), "pd_start")

    def plan(self) -> dict:
        r = PdRound()
        _check(lib().pvlm_pd_plan(self._h, _c.byref(r)), "pd_plan")
        d = {n: getattr(r, n) for n, _ in r._fields_}
        d["mode"] = _PD_MODES[r.mode]
        return d

    def finish(self, drafted, n_accepted: int, target_token=None):
        arr, n = self._arr(drafted)
        tok = -1 if target_token is None else int(target_token)
        _check(lib().pvlm_pd_finish(self._h, arr if n else None, n, int(n_accepted), tok),
               "pd_finish")

    def _tokens(self, fn):
        n = _I(0)
        _check(fn(self._h, None, 0, _c.byref(n)), "pd_tokens")
        buf = (_c.c_int32 * max(n.value, 1))()
        _check(fn(self._h, buf, n.value, _c.byref(n)), "pd_tokens")
        return list(buf[:n.value])

    def output(self):
        return self._tokens(lib().pvlm_pd_output)

    def pending(self):
        return self._tokens(lib().pvlm_pd_pending)

    def stats(self) -> dict:
        st = PdStats()
        _check(lib().pvlm_pd_get_stats(self._h, _c.byref(st)), "pd_stats")
        d = {n: getattr(st, n) for n, _ in st._fields_}
        d["mode"] = _PD_MODES[st.mode]
        return d


def rope_append(q, k_new, v_new, pos, ctx_len, k_cache, v_cache, *, base: float,
                sections=None, q_out=None, status=None):
    """pvlm_rope_append: rotate q and k_new by their positions (1-D RoPE, or
    M-RoPE with ``sections`` = (s0, s1, s2)) and write k_new / v_new into the
    caches at rows ctx_len[b] + t.  q [B][T][Hq][D]; k_new, v_new [B][T][Hkv][D];
    pos [B][T] or [3][B][T] int32; caches [B][Hkv][n_cap][D].  Returns q_out."""
    _need(q, "q")
    dev = q.device
    for t, name in ((k_new, "k_new"), (v_new, "v_new"), (k_cache, "k_cache"),
                    (v_cache, "v_cache")):
        _need(t, name, q.dtype, dev)
    _need(pos, "pos", torch.int32, dev)
    _need(ctx_len, "ctx_len", torch.int32, dev)
    B, T, Hq, D = q.shape
    Hkv = k_new.shape[2]
    n_cap = k_cache.shape[2]
    if tuple(k_new.shape) != (B, T, Hkv, D) or tuple(v_new.shape) != (B, T, Hkv, D):
        raise ValueError("k_new and v_new must be [B][T][Hkv][D]")
    if tuple(k_cache.shape) != (B, Hkv, n_cap, D) or tuple(v_cache.shape) != (B, Hkv, n_cap, D):
        raise ValueError("caches must be [B][Hkv][n_cap][D]")
    want = (B, T) if sections is None else (3, B, T)
    if tuple(pos.shape) != want:
        raise ValueError(f"pos must be {list(want)}")
    if tuple(ctx_len.shape) != (B,):
        raise ValueError("ctx_len must be [B]")
    if q_out is None:
        q_out = torch.empty_like(q)
    else:
        _need(q_out, "q_out", q.dtype, dev)
    sec = None if sections is None else (_c.c_int32 * 3)(*[int(x) for x in sections])
    st = lib().pvlm_rope_append(_dt(q), B, T, Hq, Hkv, D, n_cap, float(base), sec, _ptr(pos),
                                _ptr(q), _ptr(k_new), _ptr(v_new), _ptr(ctx_len), _ptr(q_out),
                                _ptr(k_cache), _ptr(v_cache), _ptr(_status(status)), _stream())
    _check(st, "pvlm_rope_append")
    return q_out


def rope_append_paged(q, k_new, v_new, pos, ctx_len, k_pool, v_pool, page_table, *, base: float,
                      sections=None, q_out=None, status=None):
    """pvlm_rope_append_paged: as ``rope_append``, writing the new rows into
    the pools [n_pages][Hkv][page][D] through page_table [B][max_pages]."""
    _need(q, "q")
    dev = q.device
    for t, name in ((k_new, "k_new"), (v_new, "v_new")):
        _need(t, name, q.dtype, dev)
    n_pages, Hkv, page, Dp = _pool_shape(k_pool, v_pool, page_table, dev, q.dtype)
    _need(pos, "pos", torch.int32, dev)
    _need(ctx_len, "ctx_len", torch.int32, dev)
    B, T, Hq, D = q.shape
    if tuple(k_new.shape) != (B, T, Hkv, D) or tuple(v_new.shape) != (B, T, Hkv, D) or Dp != D:
        raise ValueError("k_new and v_new must be [B][T][Hkv][D] matching the pools")
    if page_table.shape[0] != B or tuple(ctx_len.shape) != (B,):
        raise ValueError("page_table must be [B][max_pages] and ctx_len [B]")
    want = (B, T) if sections is None else (3, B, T)
    if tuple(pos.shape) != want:
        raise ValueError(f"pos must be {list(want)}")
    if q_out is None:
        q_out = torch.empty_like(q)
    else:
        _need(q_out, "q_out", q.dtype, dev)
    sec = None if sections is None else (_c.c_int32 * 3)(*[int(x) for x in sections])
    st = lib().pvlm_rope_append_paged(_dt(q), B, T, Hq, Hkv, D, page, page_table.shape[1], n_pages,
                                      float(base), sec, _ptr(pos), _ptr(q), _ptr(k_new),
                                      _ptr(v_new), _ptr(page_table), _ptr(ctx_len), _ptr(q_out),
                                      _ptr(k_pool), _ptr(v_pool), _ptr(_status(status)),
                                      _stream())
    _check(st, "pvlm_rope_append_paged")
    return q_out
