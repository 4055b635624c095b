"""The sustained FP4 MFMA probe the benchmark reports beside the roofline:
it runs, its clock reading is physical, and its rate does not exceed the
dense FP4 peak scaled to that clock (the peak is quoted at 2.4 GHz)."""

import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

pytestmark = pytest.mark.gpu


def test_mfma_probe_is_physical():
    import torch

    import bench

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    r = bench.mfma_probe(torch, dev, stream, iters=200, reps=3)
    assert 0.3 < r["clock_GHz"] < 3.0, r
    assert r["achieved"] > 0.0
    # at most the issue rate of one 32-cycle FP4 MFMA per SIMD at the measured clock (+10% for timing slack)
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    bound = cus * 4 * (2 * 32 * 32 * 64 / 32) * r["clock_GHz"] * 1e9 / 1e12
    assert r["achieved"] < 1.1 * bound, (r, bound)
