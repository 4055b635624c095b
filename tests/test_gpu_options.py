"""Options of the prepared activation and the weight, through the C ABI:
the ceil E8M0 rule (an MXFP4 ablation flag), the dense-only backbone (the
dense copy written instead of the compressed form) and the debug outputs
(keep bits per block, RMSNorm r per row).  Preparation and weight bytes must
equal the oracle's; the GEMM is checked against the oracle within the 1e-3
gate, and against the compressed-backbone GEMM bit for bit."""

import sys

import numpy as np
import pytest
import torch

from oracle import sharq_oracle as O
import panel_layout as L
from paper_2606_26587_amd import synth

pytestmark = pytest.mark.gpu

GATE = 1e-3


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


def gemm_check(y_gpu, y_ref, y_abs, tag):
    gate = O.gemm_gate_error(y_gpu, y_ref, y_abs)
    norm = float(np.abs(y_gpu.astype(np.float64) - y_ref).max() / max(np.abs(y_ref).max(), 1e-300))
    say(f"[gemm] {tag}: gate={gate:.3e} normwise={norm:.3e}")
    assert gate <= GATE and norm <= GATE, (tag, gate, norm)


def keep_bits_device(o: dict) -> np.ndarray:
    """The oracle's keep mask as the debug output's bytes: bit p of byte b of a
    row is position 8 b + p, 4 bytes per 32 positions, panel-major."""
    packed = np.packbits(o["keep"].astype(np.uint8), axis=1, bitorder="little")
    return L.to_panels(packed, o["K"])


# --------------------------------------------------------------------------- ceil E8M0 rule

@pytest.mark.parametrize("T,K,use_gamma,n,m,pairs", [(37, 416, True, 2, 4, False), (64, 4096, True, 2, 4, False),
                                                     (9, 14336, False, 2, 4, False), (33, 768, False, 4, 8, False),
                                                     (20, 1024, True, 4, 8, True), (2048, 4096, True, 2, 4, False)])
def test_ceil_rule_prep_bit_exact(S, G, T, K, use_gamma, n, m, pairs):
    say(f"[ceil-prep] T={T} K={K} {n}:{m}{'p' if pairs else ''} gamma={use_gamma}")
    x = synth.activations(T, K, seed=T + K)
    g = synth.gamma(K, seed=K) if use_gamma else None
    a = S.sharq_prepare(G.dev_bf16(x), None if g is None else G.dev_bf16(g), 1e-5, n, m, "mx", pairs=pairs,
                        scale_rule="ceil")
    torch.cuda.synchronize()
    o = O.prepare(x, g, 1e-5, n, m, "mx", pairs=pairs, scale_rule="ceil")
    f = O.prepare(x, g, 1e-5, n, m, "mx", pairs=pairs)
    assert not np.array_equal(o["sp_scale"], f["sp_scale"])   # the rule changes the scales of these inputs
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(f"ceil:{name}", G.host(getattr(a, name)), dev[name])


@pytest.mark.parametrize("N,K", [(200, 416), (6144, 4096)])
def test_ceil_rule_weight_and_gemm(S, G, N, K):
    say(f"[ceil-weight] N={N} K={K}")
    w = synth.weight(N, K, seed=N)
    q = S.sharq_quantize_weight(G.dev_bf16(w), "mx", scale_rule="ceil")
    x = synth.activations(300, K, seed=3)
    g = synth.gamma(K, seed=3)
    a = S.sharq_prepare(G.dev_bf16(x), G.dev_bf16(g), 1e-6, 2, 4, "mx", scale_rule="ceil")
    y = S.sharq_linear(a, q, dtype=torch.float32)
    torch.cuda.synchronize()
    wo = O.quantize_weight(w, "mx", scale_rule="ceil")
    dev = L.weight_to_device_layout(wo)
    G.assert_bytes_equal("codes", G.host(q.codes[0]), dev["codes"])
    G.assert_bytes_equal("scale", G.host(q.scale[0]), dev["scale"])
    o = O.prepare(x, g, 1e-6, 2, 4, "mx", scale_rule="ceil")
    gemm_check(G.host(y), O.linear(o, wo), O.linear_abs(o, wo), f"ceil N{N}K{K}")


# --------------------------------------------------------------------------- dense-only backbone

@pytest.mark.parametrize("T,K,N,use_gamma,n,m,pairs", [(2048, 4096, 6144, True, 2, 4, False),
                                                       (300, 640, 300, True, 4, 8, False),
                                                       (288, 2048, 256, False, 4, 8, True),
                                                       (16, 4096, 6144, True, 2, 4, False),
                                                       (64, 14336, 4096, False, 2, 4, False),
                                                       (5, 256, 12300, False, 4, 8, False)])
def test_dense_only_backbone(S, G, T, K, N, use_gamma, n, m, pairs):
    """The dense copy written alone: byte-exact against the oracle's backbone
    expanded to all positions, the other buffers as usual, and every GEMM that
    reads it (the persistent kernel, and the small-M kernel at M <= 256 with
    few tiles) bit-identical to the GEMM on the compressed backbone."""
    say(f"[dense-only] T={T} K={K} N={N} {n}:{m}{'p' if pairs else ''}")
    x = synth.activations(T, K, seed=K + T)
    g = synth.gamma(K, seed=3) if use_gamma else None
    xd, gd = G.dev_bf16(x), (None if g is None else G.dev_bf16(g))
    a = S.sharq_prepare(xd, gd, 1e-5, n, m, "mx", pairs=pairs,
                        out=S.alloc_act(T, K, n, m, "mx", "cuda", pairs, dense_only=True))
    c = S.sharq_prepare(xd, gd, 1e-5, n, m, "mx", pairs=pairs)
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=N)))
    yd = S.sharq_linear(a, wq, dtype=torch.float32)
    yc = S.sharq_linear(c, wq, dtype=torch.float32)
    yd16 = S.sharq_linear(a, wq, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert a.sp_codes is None and a.sp_meta is None
    o = O.prepare(x, g, 1e-5, n, m, "mx", pairs=pairs)
    dev = L.act_to_device_layout(o)
    G.assert_bytes_equal("sp_dense", G.host(a.sp_dense), L.dense_backbone_to_device_layout(o))
    for name in ("sp_scale", "dn_codes", "dn_scale"):
        G.assert_bytes_equal(name, G.host(getattr(a, name)), dev[name])
    assert torch.equal(yd, yc)
    assert torch.equal(yd16, yd.to(torch.bfloat16))
    rows = np.arange(T) if T <= 512 else np.random.default_rng(2).choice(T, 256, replace=False)
    wo = G.weight_to_oracle(wq)
    gemm_check(G.host(yd)[rows], O.linear(o, wo, rows=rows), O.linear_abs(o, wo, rows=rows), f"dense-only T{T}")


# --------------------------------------------------------------------------- debug outputs

@pytest.mark.parametrize("T,K,use_gamma,n,m,pairs,fmt,dense", [
    (37, 416, True, 2, 4, False, "mx", False), (64, 4096, True, 2, 4, False, "mx", True),
    (9, 14336, False, 2, 4, False, "mx", True), (20, 1024, True, 4, 8, False, "mx", False),
    (20, 1024, True, 4, 8, True, "nv", False), (17, 3584, True, 2, 4, False, "nv", False),
    (2048, 4096, True, 2, 4, False, "mx", True), (20, 1024, True, 4, 8, True, "nv", True),
    (9, 18944, False, 2, 4, False, "nv", True), (33, 640, True, 4, 8, False, "nv", True)])
def test_debug_outputs(S, G, T, K, use_gamma, n, m, pairs, fmt, dense):
    """The keep bits of every block and the per-row RMSNorm reciprocal r equal
    the oracle's mask and r; the prepared buffers are unchanged by the debug
    outputs."""
    say(f"[debug] T={T} K={K} {n}:{m}{'p' if pairs else ''} {fmt} gamma={use_gamma} dense={dense}")
    x = synth.activations(T, K, seed=T * 3 + K)
    g = synth.gamma(K, seed=K + 1) if use_gamma else None
    xd, gd = G.dev_bf16(x), (None if g is None else G.dev_bf16(g))
    a = S.sharq_prepare(xd, gd, 1e-6, n, m, fmt, pairs=pairs,
                        out=S.alloc_act(T, K, n, m, fmt, "cuda", pairs, dense_backbone=dense, debug=True))
    torch.cuda.synchronize()
    o = O.prepare(x, g, 1e-6, n, m, fmt, pairs=pairs)
    G.assert_bytes_equal("dbg_mask", G.host(a.dbg_mask), keep_bits_device(o))
    if use_gamma:
        assert np.array_equal(G.host(a.dbg_r).view(np.uint32), np.asarray(o["r"], np.float32).view(np.uint32))
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(f"debug:{name}", G.host(getattr(a, name)), dev[name])
    if dense:
        G.assert_bytes_equal("debug:sp_dense", G.host(a.sp_dense), L.dense_backbone_to_device_layout(o))
