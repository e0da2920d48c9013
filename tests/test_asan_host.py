"""The library's host-side code under AddressSanitizer (not gpu).

`tests/asan/host_checks.cpp` drives every entry point's argument validation,
the workspace-size queries at extreme sizes and the host-only calls (window
size, speedup model, long randomised runs of the parallel-decoding
scheduler).  It is linked against the library's sources compiled for gfx950
with AddressSanitizer on the host side only (the device code is built as
usual), so a heap or stack error, a use after free or a leak in host code
aborts the run with a report.  The build is kept under `_build/asan/` and
redone when a source changes.
"""
import concurrent.futures as cf
import hashlib
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2603_19610_amd", "csrc")
DRIVER = os.path.join(ROOT, "tests", "asan", "host_checks.cpp")
OUT = os.path.join(ROOT, "_build", "asan")
HIPCC = "/opt/rocm/bin/hipcc"
COMMON = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-Xarch_host", "-fsanitize=address",
          "-I" + os.path.join(ROOT, "include")]


def _sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


def _digest():
    h = hashlib.sha256()
    for p in _sources() + [DRIVER, os.path.join(CSRC, "common.h"), os.path.join(ROOT, "include", "pvlm.h")]:
        h.update(open(p, "rb").read())
    return h.hexdigest()


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(" ".join(cmd) + "\n" + r.stderr[-4000:])


def _build():
    exe = os.path.join(OUT, "host_checks")
    stamp = os.path.join(OUT, "digest")
    d = _digest()
    if os.path.exists(exe) and os.path.exists(stamp) and open(stamp).read() == d:
        return exe
    os.makedirs(OUT, exist_ok=True)
    objs, cmds = [], []
    for src in _sources():
        o = os.path.join(OUT, os.path.basename(src)[:-4] + ".o")
        objs.append(o)
        cmds.append([HIPCC, "--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang",
                     "-packed-fp32-ops", *COMMON, "-I" + CSRC, "-c", src, "-o", o])
    drv = os.path.join(OUT, "host_checks.o")
    cmds.append([HIPCC, "-x", "c++", *COMMON, "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", "-c",
                 DRIVER, "-o", drv])
    with cf.ThreadPoolExecutor(max_workers=min(4, os.cpu_count() or 1)) as ex:
        list(ex.map(_run, cmds))
    _run([HIPCC, "-Xarch_host", "-fsanitize=address", "-o", exe, drv, *objs])
    open(stamp, "w").write(d)
    return exe


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_host_code_under_address_sanitizer():
    exe = _build()
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:exitcode=3")
    r = subprocess.run([exe], capture_output=True, text=True, timeout=600, env=env)
    assert "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
    assert r.returncode == 0, r.stdout + r.stderr[-4000:]
    assert "host checks: ok" in r.stdout
