"""Host-side logic of bench.py, without a GPU: the work and byte counts the
JSON line reports, the one-GPU guard, and the traffic record's shape."""

import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def test_flop_counts():
    T, N, K = 2048, 6144, 4096
    # executed: backbone (run dense) + residual, 2 T N K each
    assert bench.gemm_flops(T, N, K) == 4.0 * T * N * K
    # algorithmic: residual 2 T N K + backbone over n of m positions
    assert bench.alg_flops(T, N, K, 2, 4) == 3.0 * T * N * K
    assert bench.alg_flops(T, N, K, 4, 8) == 3.0 * T * N * K
    assert bench.alg_flops(T, N, K, 1, 4) == 2.5 * T * N * K
    assert bench.lin_flops(T, N, K) == 2.0 * T * N * K


def test_prep_bytes():
    T, K = 2048, 4096
    # MXFP4 2:4: bf16 X and gamma in; K/4 backbone codes, K/8 metadata,
    # K/32 + K/32 scales, K/2 residual codes out
    assert bench.prep_bytes(T, K, True) == 2 * T * K + 2 * K + T * (K / 4 + K / 8 + K / 16 + K / 2)
    assert bench.prep_bytes(T, K, False) == 2 * T * K + T * (K / 4 + K / 8 + K / 16 + K / 2)
    # NVFP4: the residual keeps one E4M3 scale per 16
    assert bench.prep_bytes(T, K, False, fmt="nv") - bench.prep_bytes(T, K, False) == T * K / 32
    # the dense copy alone replaces codes + metadata (3K/8) by K/2
    assert bench.prep_bytes_written(T, K, True, backbone="dense-only") - bench.prep_bytes(T, K, True) == T * K / 8
    assert bench.prep_bytes_written(T, K, True, backbone="both") - bench.prep_bytes(T, K, True) == T * K / 2


def test_traffic_record():
    d = bench.gemm_source_digest()
    assert len(d) == 16 and int(d, 16) >= 0
    assert set(bench.TRAFFIC) == {"gemm_source", "bytes_per_launch"}
    assert bench.TRAFFIC["bytes_per_launch"] > 0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_warmup_tenths():
    assert bench.tenths([]) == []
    assert bench.tenths([2.0]) == [2.0]
    assert bench.tenths([1.0, 3.0, 5.0]) == [1.0, 3.0, 5.0]
    t = bench.tenths(list(range(200)))
    assert len(t) == 10 and t[0] == 9.5 and t[-1] == 189.5
