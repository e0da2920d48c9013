"""bench.py's contract on the CPU (not gpu): it refuses more than one GPU
before touching a device, and the verify roofline's algorithmic bytes per
launch at the LLaVA-OV-72B layer shape are the ones the roofline quotes,
recomputed here from the shape."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr or "one MI355X" in r.stderr
    assert r.stdout.strip() == ""


def test_verify_bytes_at_72b_shape():
    sys.path.insert(0, ROOT)
    import bench
    import workloads as W
    w = W.WORKLOADS["llava72b"]
    T = w.gamma + 1
    N = 64 * 196 + 256 + T                    # visual + text + verify rows
    kv = 2 * N * 8 * 128 * 2                  # K and V, 8 KV heads, D 128, bf16
    q_o = 2 * T * 64 * 128 * 2                # Q in, O out
    mass, lse = 4 * N, 4 * 64 * T
    assert bench.verify_bytes(w) == kv + q_o + mass + lse == 52_814_116
