"""The preparation and the two-path GEMM in one call (sharq_prepare_linear),
through the C ABI: for a few rows one kernel prepares the rows in its
prologue.  The prepared activation it writes must equal the oracle's byte for
byte, Y must match the oracle within the 1e-3 gate and equal the separate
sharq_prepare + sharq_linear bit for bit."""

import sys

import numpy as np
import pytest
import torch

from oracle import sharq_oracle as O
import panel_layout as L
from paper_2606_26587_amd import synth

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def S():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2606_26587_amd import sharq
    return sharq


@pytest.fixture(scope="module")
def G(S):
    import gpu_util
    return gpu_util


def say(*a):
    print(*a, file=sys.stderr, flush=True)


CASES = [  # (M, K, N, gamma, n, m, pairs, backbone)
    (1, 4096, 6144, True, 2, 4, False, "compressed"), (1, 4096, 28672, True, 2, 4, False, "dense-only"),
    (1, 14336, 4096, False, 2, 4, False, "both"), (2, 4096, 6144, True, 4, 8, False, "compressed"),
    (3, 1024, 300, True, 2, 4, False, "both"), (4, 4096, 6144, True, 2, 4, False, "dense-only"),
    (4, 2048, 1536, True, 4, 8, True, "compressed"), (1, 128, 40, True, 2, 4, False, "compressed"),
    (6, 4096, 6144, True, 2, 4, False, "compressed"), (16, 4096, 6144, True, 2, 4, False, "dense-only")]


@pytest.mark.parametrize("M,K,N,use_gamma,n,m,pairs,backbone", CASES)
@pytest.mark.parametrize("ydt", [torch.float32, torch.bfloat16])
def test_prepare_linear(S, G, M, K, N, use_gamma, n, m, pairs, backbone, ydt):
    say(f"[fused] M={M} K={K} N={N} {n}:{m}{'p' if pairs else ''} gamma={use_gamma} {backbone} {ydt}")
    x = synth.activations(M, K, seed=M + K)
    g = synth.gamma(K, seed=K) if use_gamma else None
    xd, gd = G.dev_bf16(x), (None if g is None else G.dev_bf16(g))
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=N)))

    def act():
        return S.alloc_act(M, K, n, m, "mx", "cuda", pairs, dense_backbone=backbone == "both",
                           dense_only=backbone == "dense-only", debug=True)

    a, y = S.sharq_prepare_linear(xd, gd, wq, 1e-5, n, m, "mx", act=act(), dtype=ydt, pairs=pairs)
    b = S.sharq_prepare(xd, gd, 1e-5, n, m, "mx", pairs=pairs, out=act())
    y2 = S.sharq_linear(b, wq, dtype=ydt)
    torch.cuda.synchronize()
    assert torch.equal(y, y2)
    for name in ("sp_codes", "sp_meta", "sp_dense", "sp_scale", "dn_codes", "dn_scale", "dbg_mask"):
        t1, t2 = getattr(a, name), getattr(b, name)
        if t1 is None:
            assert t2 is None
            continue
        G.assert_bytes_equal(name, G.host(t1), G.host(t2))
    if use_gamma:
        assert torch.equal(a.dbg_r, b.dbg_r)
    o = O.prepare(x, g, 1e-5, n, m, "mx", pairs=pairs)
    dev = L.act_to_device_layout(o)
    for name in ("sp_scale", "dn_codes", "dn_scale"):
        G.assert_bytes_equal(name, G.host(getattr(a, name)), dev[name])
    if a.sp_codes is not None:
        G.assert_bytes_equal("sp_codes", G.host(a.sp_codes), dev["sp_codes"])
        G.assert_bytes_equal("sp_meta", G.host(a.sp_meta), dev["sp_meta"])
    if a.sp_dense is not None:
        G.assert_bytes_equal("sp_dense", G.host(a.sp_dense), L.dense_backbone_to_device_layout(o))
    if ydt == torch.float32:
        wo = G.weight_to_oracle(wq)
        gate = O.gemm_gate_error(G.host(y), O.linear(o, wo), O.linear_abs(o, wo))
        say(f"[fused] gate={gate:.3e}")
        assert gate <= 1e-3


def test_prepare_linear_rejects_before_launch(S, G):
    """A bad GEMM argument is reported before the preparation runs: the
    prepared activation stays untouched."""
    M, K, N = 1, 256, 64
    x = G.dev_bf16(synth.activations(M, K, seed=1))
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=1)))
    a = S.alloc_act(M, K, 2, 4, "mx", "cuda")
    a.dn_codes.fill_(0xAB)
    y = torch.empty((M, N), dtype=torch.float32, device="cuda")
    with pytest.raises(S.SharqError):
        S.sharq_prepare_linear(x, None, wq, 1e-6, act=a, out=y.double())   # fp64 output: not supported
    torch.cuda.synchronize()
    assert torch.all(a.dn_codes == 0xAB)
