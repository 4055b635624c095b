"""SiLU.mul fused into the preparation of the down projection's input
(producer-side fusion, Sec. 4.3), through the C ABI, against the CPU oracle.

h = bf16(SiLU(g) * u) follows one fp32 recipe on both sides (an exponential
by Cody-Waite reduction and a Taylor polynomial, correctly rounded division),
so h must equal the oracle's byte for byte, and so must everything after it
(mask, codes, metadata, scales, the NVFP4 per-tensor scale)."""

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


def check_silu(S, G, T, K, n, m, fmt, pairs, tag, strided=False, seed=0):
    say(f"[silu] {tag} T={T} K={K} {n}:{m}{'p' if pairs else ''} {fmt} strided={strided}")
    gate = synth.activations(T, K, seed=seed + 1)
    up = synth.activations(T, K, seed=seed + 2)
    if strided:   # the two halves of one [T, 2K] gate/up output
        gu = G.dev_bf16(np.concatenate([gate, up], axis=1))
        gd, ud = gu[:, :K], gu[:, K:]
    else:
        gd, ud = G.dev_bf16(gate), G.dev_bf16(up)
    h = torch.empty((T, K), dtype=torch.bfloat16, device="cuda")
    a = S.sharq_prepare_silu_mul(gd, ud, n, m, fmt, h_out=h, pairs=pairs)
    b = S.sharq_prepare_silu_mul(gd, ud, n, m, fmt, pairs=pairs)     # without writing h
    torch.cuda.synchronize()
    h_gpu = G.host(h.view(torch.int16)).view(np.uint16)
    o = O.prepare_silu_mul(gate, up, n, m, fmt, pairs=pairs)
    G.assert_bytes_equal(f"{tag}:h", h_gpu, o["h"])
    if fmt == "nv":
        for act in (a, b):
            got = np.asarray(G.host(act.tensor_scale)[0], np.float32).view(np.uint32)
            assert got == np.asarray(o["tensor_scale"], np.float32).view(np.uint32), tag
    dev = L.act_to_device_layout(o)
    for act in (a, b):
        for name in O.ACT_BUFFERS:
            G.assert_bytes_equal(f"{tag}:{name}", G.host(getattr(act, name)), dev[name])


@pytest.mark.parametrize("T,K,n,m,pairs,fmt,strided", [
    (8, 128, 2, 4, False, "mx", False),
    (37, 416, 2, 4, False, "mx", True),
    (19, 640, 4, 8, False, "mx", False),
    (23, 1024, 4, 8, True, "nv", True),
    (33, 3584, 2, 4, False, "nv", False),
    (1, 14336, 2, 4, False, "mx", False),
])
def test_silu_mul_prep(S, G, T, K, n, m, pairs, fmt, strided):
    check_silu(S, G, T, K, n, m, fmt, pairs, f"T{T}K{K}", strided=strided, seed=T)


def test_silu_mul_edge_values(S, G):
    """Gate values where the recipe's exponential underflows into fp32
    subnormals or to zero, signed zeros, tiny and huge products: h byte for
    byte, and the preparation of h."""
    T, K = 6, 256
    rng = np.random.default_rng(44)
    specials = np.array([0.0, -0.0, 1e-30, -1e-30, -87.0, -88.5, -95.0, -103.0, -103.9, -104.5, -120.0, -200.0,
                         20.0, 88.0, 100.0, -5.0], np.float32)
    g = rng.choice(specials, size=(T, K)).astype(np.float32)
    u = (rng.standard_normal((T, K)) * 10.0 ** rng.integers(-30, 30, size=(T, K))).astype(np.float32)
    u[0, :16] = [1e30, -1e30, 3e35, 1e-38, 0.0, -0.0, 1.0, -1.0, 5e34, 2e-20, 7.0, 1e10, -1e25, 1e35, 1e-30, 2.0]
    gate, up = synth.f32_to_bf16_bits(g), synth.f32_to_bf16_bits(u)
    h = torch.empty((T, K), dtype=torch.bfloat16, device="cuda")
    a = S.sharq_prepare_silu_mul(G.dev_bf16(gate), G.dev_bf16(up), 2, 4, "mx", h_out=h)
    torch.cuda.synchronize()
    o = O.prepare_silu_mul(gate, up, 2, 4, "mx")
    G.assert_bytes_equal("h", G.host(h.view(torch.int16)).view(np.uint16), o["h"])
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(name, G.host(getattr(a, name)), dev[name])


def test_silu_mul_llama_down_full_shape(S, G):
    """The Llama-3.1-8B down projection's input at M = 2048 (K = 14336), from a
    [2048, 28672] gate/up output, compared in full."""
    check_silu(S, G, 2048, 14336, 2, 4, "mx", False, "llama-down", strided=True, seed=5)


def test_silu_mul_then_linear(S, G):
    """The fused preparation feeds the GEMM like any prepared activation."""
    T, K, N = 64, 1024, 256
    gate, up = synth.activations(T, K, seed=7), synth.activations(T, K, seed=8)
    h = torch.empty((T, K), dtype=torch.bfloat16, device="cuda")
    a = S.sharq_prepare_silu_mul(G.dev_bf16(gate), G.dev_bf16(up), 2, 4, "mx", h_out=h)
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=7)))
    y = S.sharq_linear(a, wq, dtype=torch.float32)
    torch.cuda.synchronize()
    o = O.prepare(G.host(h.view(torch.int16)).view(np.uint16), None, 0.0, 2, 4, "mx")
    wo = G.weight_to_oracle(wq)
    ref, absd = O.linear(o, wo), O.linear_abs(o, wo)
    assert O.gemm_gate_error(G.host(y), ref, absd) <= 1e-3


def test_silu_mul_empty(S, G):
    e = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    a = S.sharq_prepare_silu_mul(e, e, 2, 4, "mx")
    torch.cuda.synchronize()
    assert a.rows == 0


@pytest.mark.parametrize("T,K,n,m,pairs", [(33, 3584, 2, 4, False), (23, 1024, 4, 8, True)])
def test_silu_mul_prep_nv_dense_only(S, G, T, K, n, m, pairs):
    """NVFP4 SiLU.mul preparation with the backbone as its dense copy alone:
    the copy and the other buffers byte-exact against the oracle."""
    say(f"[silu] nv dense-only T={T} K={K} {n}:{m}{'p' if pairs else ''}")
    gate = synth.activations(T, K, seed=T + 11)
    up = synth.activations(T, K, seed=T + 12)
    a = S.sharq_prepare_silu_mul(G.dev_bf16(gate), G.dev_bf16(up), n, m, "nv", pairs=pairs,
                                 out=S.alloc_act(T, K, n, m, "nv", "cuda", pairs, dense_only=True))
    torch.cuda.synchronize()
    o = O.prepare_silu_mul(gate, up, n, m, "nv", pairs=pairs)
    got = np.asarray(G.host(a.tensor_scale)[0], np.float32).view(np.uint32)
    assert got == np.asarray(o["tensor_scale"], np.float32).view(np.uint32)
    G.assert_bytes_equal("sp_dense", G.host(a.sp_dense), L.dense_backbone_to_device_layout(o))
    dev = L.act_to_device_layout(o)
    for name in ("sp_scale", "dn_codes", "dn_scale"):
        G.assert_bytes_equal(name, G.host(getattr(a, name)), dev[name])
