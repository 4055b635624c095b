"""The sustained MFMA probes the benchmark reports beside the rooflines
(scaled FP4, bf16 and fp16): each runs, its clock reading is physical, and its rate
does not exceed the dense peak of its instruction scaled to that clock (the
peaks are quoted at 2.4 GHz)."""

import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("kind,flops_per_mfma", [("fp4", 2 * 32 * 32 * 64), ("bf16", 2 * 32 * 32 * 16),
                                                   ("f16", 2 * 32 * 32 * 16)])
def test_mfma_probe_is_physical(kind, flops_per_mfma):
    import torch

    import bench

    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    r = bench.mfma_probe(torch, dev, stream, iters=200, reps=3, kind=kind)
    assert 0.3 < r["clock_GHz"] < 3.0, r
    assert r["achieved"] > 0.0
    # at most one 32-cycle MFMA per SIMD at the measured clock (+10% for
    # timing slack): 4096 (FP4) and 1024 (bf16, fp16) flops per cycle per SIMD are
    # the published peaks at 2.4 GHz on 1024 SIMDs
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    bound = cus * 4 * (flops_per_mfma / 32) * r["clock_GHz"] * 1e9 / 1e12
    assert r["achieved"] < 1.1 * bound, (r, bound)
