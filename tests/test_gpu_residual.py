"""Residual add fused into the preparation (sharq_prepare_residual) on the
HIP path, through the C ABI, against the CPU oracle: h = bf16(x + res) and
every prepared buffer byte for byte, out of place and in place."""

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


def f32_bits(v) -> int:
    return int(np.asarray(v, dtype=np.float32).view(np.uint32))


def check(S, G, x, res, g, eps, n, m, fmt, pairs, tag, in_place=False):
    say(f"[residual] {tag} {fmt} {n}:{m}{'p' if pairs else ''} shape={x.shape} gamma={g is not None} "
        f"in_place={in_place}")
    xd, rd = G.dev_bf16(x), G.dev_bf16(res)
    a, h = S.sharq_prepare_residual(xd, rd, None if g is None else G.dev_bf16(g), eps, n, m, fmt,
                                    h_out=rd if in_place else None, pairs=pairs)
    torch.cuda.synchronize()
    o = O.prepare_residual(x, res, g, eps, n, m, fmt, pairs=pairs)
    G.assert_bytes_equal(f"{tag}:h", G.host(h.view(torch.int16)).view(np.uint16), o["h"])
    if in_place:
        assert h.data_ptr() == rd.data_ptr()
    else:
        G.assert_bytes_equal(f"{tag}:residual untouched", G.host(rd.view(torch.int16)).view(np.uint16), res)
    if fmt == "nv":
        assert f32_bits(G.host(a.tensor_scale)[0]) == f32_bits(o["tensor_scale"]), tag
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(f"{tag}:{name}", G.host(getattr(a, name)), dev[name])


CASES = [
    # (T, K, gamma, n, m, fmt, pairs): every preparation kernel shape class
    (8, 128, True, 2, 4, "mx", False),
    (37, 416, True, 2, 4, "mx", False),      # ragged last panel
    (64, 4096, True, 2, 4, "mx", False),     # two wavefronts per row
    (9, 16384, True, 2, 4, "mx", False),     # several blocks per lane
    (33, 14336, False, 2, 4, "mx", False),   # one thread per block, no norm
    (130, 2048, True, 4, 8, "mx", False),
    (17, 3584, True, 2, 4, "nv", False),     # NVFP4: the amax pre-pass forms h too
    (6, 18944, False, 2, 4, "nv", False),
    (40, 4096, True, 4, 8, "nv", True),      # 4:8 in pairs
]


@pytest.mark.parametrize("T,K,use_gamma,n,m,fmt,pairs", CASES)
def test_prepare_residual_bit_exact(S, G, T, K, use_gamma, n, m, fmt, pairs):
    x = synth.activations(T, K, seed=T + K)
    res = synth.activations(T, K, seed=T + 2 * K + 1)
    g = synth.gamma(K, seed=K) if use_gamma else None
    check(S, G, x, res, g, 1e-5, n, m, fmt, pairs, f"T{T}K{K}")


@pytest.mark.parametrize("use_gamma", [True, False])
def test_prepare_residual_in_place(S, G, use_gamma):
    """h_out = residual: the residual stream is updated in place (rows of a
    partial last row group included)."""
    T, K = 45, 4096
    x = synth.activations(T, K, seed=41)
    res = synth.activations(T, K, seed=42)
    g = synth.gamma(K, seed=4) if use_gamma else None
    check(S, G, x, res, g, 1e-5, 2, 4, "mx", False, "in-place", in_place=True)


def test_prepare_residual_cancellation_and_ties(S, G):
    """x = -res (h all zero rows), exact bf16 ties, equal magnitudes."""
    T, K = 12, 256
    rng = np.random.default_rng(5)
    v = rng.integers(-4, 5, size=(T, K)).astype(np.float32)
    x = (v.view(np.uint32) >> 16).astype(np.uint16)
    res = x ^ np.uint16(0x8000)                    # x + res = 0
    res[3:] = np.uint16(0x3B80)                    # 2^-8: ties against the integers
    check(S, G, x, res, synth.gamma(K, seed=5), 1e-6, 2, 4, "mx", False, "ties")
    check(S, G, x, res, None, 1e-6, 2, 4, "mx", False, "ties-plain")


@pytest.mark.parametrize("T,K,use_gamma,n,m,pairs", [(17, 3584, True, 2, 4, False), (40, 4096, True, 4, 8, True),
                                                     (6, 18944, False, 2, 4, False)])
def test_prepare_residual_nv_dense_only(S, G, T, K, use_gamma, n, m, pairs):
    """NVFP4 with the backbone as its dense copy alone: h, the per-tensor
    scale, the copy and the other buffers byte-exact against the oracle."""
    say(f"[residual] nv dense-only T={T} K={K} {n}:{m}{'p' if pairs else ''}")
    x = synth.activations(T, K, seed=T + K + 5)
    res = synth.activations(T, K, seed=T + 2 * K + 6)
    g = synth.gamma(K, seed=K + 1) if use_gamma else None
    a, h = S.sharq_prepare_residual(G.dev_bf16(x), G.dev_bf16(res), None if g is None else G.dev_bf16(g), 1e-5,
                                    n, m, "nv", pairs=pairs,
                                    out=S.alloc_act(T, K, n, m, "nv", "cuda", pairs, dense_only=True))
    torch.cuda.synchronize()
    o = O.prepare_residual(x, res, g, 1e-5, n, m, "nv", pairs=pairs)
    G.assert_bytes_equal("h", G.host(h.view(torch.int16)).view(np.uint16), o["h"])
    assert f32_bits(G.host(a.tensor_scale)[0]) == f32_bits(o["tensor_scale"])
    G.assert_bytes_equal("sp_dense", G.host(a.sp_dense), L.dense_backbone_to_device_layout(o))
    dev = L.act_to_device_layout(o)
    for name in ("sp_scale", "dn_codes", "dn_scale"):
        G.assert_bytes_equal(name, G.host(getattr(a, name)), dev[name])
