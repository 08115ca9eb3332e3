"""Host-side checks of bench.py's contract that need no GPU."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    """This build measures one GPU's TP share: --gpus N > 1 exits with a message."""
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout.strip() == ""


def test_algorithmic_bytes():
    """The roofline's algorithmic bytes per launch: packed codes, scales,
    zeros, X and Y (and g_idx on the act-order path), for the Llama-70B TP=8
    GEMM1 shard at M = 16."""
    sys.path.insert(0, ROOT)
    import bench
    K, N, G, M = 8192, 3584, 128, 16
    codes, scales, zeros = K * N // 2, (K // G) * N * 2, (K // G) * N // 2
    x, y = M * K * 2, M * N * 2
    assert bench.gemm_bytes(M, K, N, G) == codes + scales + zeros + x + y
    assert bench.gemm_bytes(M, K, N, G, gidx=True) == codes + scales + zeros + x + y + K * 4


def test_traffic_summary_is_parsed():
    """The committed counter summary carries a source hash and a per-launch
    byte count that bench.py can read."""
    path = os.path.join(ROOT, "profiles", "traffic_decode_ordered_llama70b_tp8_M16.txt")
    text = open(path).read()
    assert "kernel_source_hash = " in text and "bytes_per_launch = " in text
    json.dumps(text)  # plain text, nothing to execute


def test_mfma_counter_summary_is_parsed():
    """The committed prefill counter summary gives each GEMM's MFMA-busy
    fraction of its clocks and the clock it ran at, both in range."""
    sys.path.insert(0, ROOT)
    import bench
    u = bench.read_mfma_util()
    assert u is not None
    for g in ("gemm1", "gemm2"):
        assert 0.0 < u[g]["mfma_busy_of_clocks"] <= 1.0
        assert 1.0 < u[g]["clock_ghz"] < 3.0
