"""C-ABI checks that need no GPU: the library loads, exports every symbol
include/pvlm.h declares, and rejects bad host arguments before launching."""
import ctypes
import os
import re

import pytest

import paper_2603_19610_amd as pv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
FAKE = ctypes.c_void_p(4096)   # never dereferenced: every case fails host validation


def _declared():
    src = open(os.path.join(ROOT, "include", "pvlm.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(pvlm_[a-z0-9_]+)\s*\(", src)))


def test_every_declared_symbol_is_exported():
    L = pv.lib()
    names = _declared()
    assert len(names) >= 13
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(pv.EXPORTS)
    assert L.pvlm_version() == 1
    assert L.pvlm_status_string(0) == b"ok"


def _verify(**kw):
    a = dict(dt=1, B=1, T=5, Hq=8, Hkv=2, D=128, n_cap=100, max_ctx=95, scale=0.088,
             q=FAKE, k=FAKE, v=FAKE, ctx=FAKE, out=FAKE, ws=FAKE, ws_bytes=1 << 30)
    a.update(kw)
    return pv.lib().pvlm_verify_attn(a["dt"], a["B"], a["T"], a["Hq"], a["Hkv"], a["D"],
                                     a["n_cap"], a["max_ctx"], a["scale"], a["q"], a["k"], a["v"],
                                     a["ctx"], a["out"], None, None, a["ws"], a["ws_bytes"],
                                     None, None)


@pytest.mark.parametrize("kw,code", [
    (dict(q=None), 1), (dict(ctx=None), 1), (dict(out=None), 1),
    (dict(T=0), 2), (dict(B=0), 2), (dict(max_ctx=96), 2), (dict(max_ctx=-1), 2),
    (dict(scale=0.0), 2), (dict(scale=float("nan")), 2),
    (dict(D=96), 3), (dict(Hkv=3), 3), (dict(T=33), 3), (dict(dt=7), 3),
    (dict(Hq=128, Hkv=1, T=9, max_ctx=90), 3),
])
def test_verify_rejects(kw, code):
    assert _verify(**kw) == code


def test_other_calls_reject():
    L = pv.lib()
    # topk: NULL score, bad B
    assert L.pvlm_topk_select(1, 10, FAKE, FAKE, 4, None, FAKE, None, 0, None, None) == 1
    assert L.pvlm_topk_select(0, 10, FAKE, FAKE, 4, FAKE, FAKE, None, 0, None, None) == 2
    # gather: unsupported row size, NULL destination
    assert L.pvlm_gather_kv(1, 1, 1, 1, 3, 10, FAKE, FAKE, FAKE, FAKE, 4, FAKE, FAKE, 8, FAKE,
                            FAKE, None, None) == 3
    assert L.pvlm_gather_kv(1, 1, 1, 1, 128, 10, FAKE, FAKE, FAKE, FAKE, 4, FAKE, FAKE, 8, None,
                            FAKE, None, None) == 1
    assert L.pvlm_gather_kv(1, 0, 1, 1, 128, 10, FAKE, FAKE, FAKE, FAKE, 4, FAKE, FAKE, 8, FAKE,
                            FAKE, None, None) == 2
    # accept: gamma 0, too many rows, negative temperature, tiny workspace
    args = [FAKE] * 8
    assert L.pvlm_spec_accept(1, 0, 10, 1.0, *args, FAKE, 1 << 20, None, None) == 2
    assert L.pvlm_spec_accept(300, 2, 10, 1.0, *args, FAKE, 1 << 20, None, None) == 3
    assert L.pvlm_spec_accept(1, 2, 10, -1.0, *args, FAKE, 1 << 20, None, None) == 2
    assert L.pvlm_spec_accept(1, 2, 10, 1.0, *args, FAKE, 8, None, None) == 4
    # uvprune: MASS with L = 0, COSSIM with a hidden size that is not a multiple of 8
    assert L.pvlm_uvprune_score(0, 1, 0, 10, FAKE, FAKE, 0, 0, 0, None, None, None, FAKE, None, 0,
                                None, None) == 2
    assert L.pvlm_uvprune_score(1, 1, 2, 10, FAKE, None, 1, 7, 4, FAKE, FAKE, FAKE, FAKE, FAKE,
                                1 << 20, None, None) == 2
    assert L.pvlm_uvprune_score(1, 1, 2, 10, FAKE, None, 1, 8, 4, FAKE, FAKE, FAKE, FAKE, FAKE,
                                4, None, None) == 4
    assert L.pvlm_spec_accept_workspace_size(1, 8, 152064) > 0
    assert L.pvlm_uvprune_workspace_size(0, 1, 8192, 256) == 0


def test_product_path_never_uses_the_oracle():
    pkg = os.path.join(ROOT, "paper_2603_19610_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle", text, re.M), f
                assert "oracle/" not in text, f


def test_missing_library_fails_loudly(monkeypatch):
    monkeypatch.setattr(pv, "_lib", None)
    monkeypatch.setattr(pv, "LIB_PATH", "/nonexistent/libpvlm.so")
    with pytest.raises(RuntimeError, match="not built"):
        pv.lib()


def test_paged_calls_reject():
    """Host-side argument checks of the paged entry points (nothing launched)."""
    L = pv.lib()

    def verify(dt=1, page=32, max_pages=4, n_pages=8, table=FAKE):
        return L.pvlm_verify_attn_paged(dt, 1, 5, 8, 2, 128, page, max_pages, n_pages, 100, 0.088,
                                        FAKE, FAKE, FAKE, table, FAKE, FAKE, None, None, FAKE,
                                        1 << 30, None, None)
    assert verify(table=None) == 1
    for bad in (dict(page=48), dict(page=16), dict(page=1 << 21), dict(max_pages=0),
                dict(n_pages=0), dict(n_pages=1 << 31)):
        assert verify(**bad) == 2, bad
    assert verify(dt=0) == 3                          # bf16 only
    assert verify(max_pages=3) == 2                   # 96 logical rows < max_ctx + T

    def gather(page=64, table=FAKE):
        return L.pvlm_gather_kv_paged(1, 2, 1, 1, 128, page, 4, 8, FAKE, FAKE, table, FAKE, FAKE,
                                      4, FAKE, FAKE, 8, FAKE, FAKE, None, None)
    assert gather(table=None) == 1
    assert gather(page=100) == 2

    def rope(B=1, page=32, table=FAKE):
        return L.pvlm_rope_append_paged(1, B, 4, 8, 2, 128, page, 4, 8, 1e6, None, FAKE, FAKE,
                                        FAKE, FAKE, table, FAKE, FAKE, FAKE, FAKE, None, None)
    assert rope(table=None) == 1
    assert rope(page=24) == 2


def test_rope_rejects_more_pairs_than_one_launch_holds():
    L = pv.lib()
    # B * T * (Hq + 2 Hkv) * D / 2 = 4096 * 32 * 80 * 512 > 2^32 - 256
    assert L.pvlm_rope_append(1, 4096, 32, 64, 8, 1024, 64, 1e6, None, FAKE, FAKE, FAKE, FAKE,
                              FAKE, FAKE, FAKE, FAKE, None, None) == 2


def test_uvprune_rejects_more_work_items_than_one_launch_holds():
    L = pv.lib()
    # MASS: B * m_cap = 8 * 2^30 scores > 2^32 - 256 work-items
    assert L.pvlm_uvprune_score(0, 8, 1, 1 << 30, FAKE, FAKE, 0, 0, 0, None, None, None, FAKE,
                                None, 0, None, None) == 2
    # COSSIM: 64 lanes * 2 * B * n_cap = 64 * 2 * 17 * (2^21 - 32) > 2^32 - 256, while
    # 2 * B stays within the grid's y
    assert L.pvlm_uvprune_score(1, 17, 2, 10, FAKE, None, 1, 8, (1 << 21) - 32, FAKE, FAKE, FAKE,
                                FAKE, FAKE, 1 << 40, None, None) == 2
    assert L.pvlm_uvprune_score(1, 8, 2, 10, FAKE, None, 1, 8, (1 << 21) - 32, FAKE, FAKE, FAKE,
                                FAKE, FAKE, 8, None, None) == 4   # within the limits: ws too small
