"""4:8 in pairs -- the NVFP4 sparsity pattern of the paper's primary
instantiation (App. A.1.4; Fig. 2 "pair-topk 4:8 in-pairs mask") -- on the HIP
path, through the C ABI, against the CPU oracle.

Preparation must match byte for byte (including the per-tensor scale bits
for NVFP4); the two-path GEMM, which reads the same keep-mask metadata as
plain 4:8, must meet the 1e-3 accumulation gate.
"""

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


def f32_bits(v) -> int:
    return int(np.asarray(v, dtype=np.float32).view(np.uint32))


def check_prep_pairs(S, G, x, g, eps, fmt, tag):
    say(f"[pairs-prep] {tag} {fmt} shape={x.shape} gamma={g is not None}")
    a = S.sharq_prepare(G.dev_bf16(x), None if g is None else G.dev_bf16(g), eps, 4, 8, fmt, pairs=True)
    torch.cuda.synchronize()
    o = O.prepare(x, g, eps, 4, 8, fmt, pairs=True)
    if fmt == "nv":
        assert f32_bits(G.host(a.tensor_scale)[0]) == f32_bits(o["tensor_scale"]), tag
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(f"{tag}:{name}", G.host(getattr(a, name)), dev[name])
    return a, o


PREP_CASES = [
    # (T, K, gamma, eps): several panels, a ragged last panel, both prep kernels
    (8, 128, True, 1e-6),
    (37, 416, True, 1e-5),
    (37, 416, False, 1e-5),
    (130, 2048, True, 1e-6),
    (64, 4096, True, 1e-5),
    (9, 14336, False, 1e-5),
    (6, 18944, False, 1e-6),
    (17, 3584, True, 1e-6),
]


@pytest.mark.parametrize("fmt", ["nv", "mx"])
@pytest.mark.parametrize("T,K,use_gamma,eps", PREP_CASES)
def test_pairs_prep_bit_exact(S, G, fmt, T, K, use_gamma, eps):
    x = synth.activations(T, K, seed=T + 7 * K)
    g = synth.gamma(K, seed=K + 2) if use_gamma else None
    check_prep_pairs(S, G, x, g, eps, fmt, f"T{T}K{K}")


@pytest.mark.parametrize("fmt", ["nv", "mx"])
def test_pairs_prep_ties(S, G, fmt):
    """Small integers: equal magnitudes inside and across pairs, so the
    tie rule (lower pair wins) decides most groups."""
    rng = np.random.default_rng(21)
    v = rng.integers(-3, 4, size=(40, 256)).astype(np.float32)
    v[:, ::8] = v[:, 1::8]          # equal elements inside a pair
    v[5] = 2.0                      # every score equal
    v[6] = 0.0                      # all-zero row
    x = (v.view(np.uint32) >> 16).astype(np.uint16)
    check_prep_pairs(S, G, x, None, 1e-6, fmt, "ties")
    check_prep_pairs(S, G, x, synth.gamma(256, seed=3), 1e-6, fmt, "ties-norm")


def gemm_check(y, ref, absref, tag):
    gate = O.gemm_gate_error(y, ref, absref)
    rel = float(np.abs(np.asarray(y, np.float64) - ref).max() / max(np.abs(ref).max(), 1e-30))
    say(f"  {tag}: gate {gate:.2e} normwise {rel:.2e}")
    assert gate <= GATE, (tag, gate)
    assert rel <= GATE, (tag, rel)


@pytest.mark.parametrize("fmt", ["nv", "mx"])
@pytest.mark.parametrize("T,N,K", [(8, 64, 128), (129, 300, 640), (256, 512, 2048), (300, 200, 416)])
def test_pairs_linear_parity(S, G, fmt, T, N, K):
    say(f"[pairs-linear] {fmt} T={T} N={N} K={K}")
    x = synth.activations(T, K, seed=T + N)
    a, o = check_prep_pairs(S, G, x, synth.gamma(K, seed=1), 1e-6, fmt, f"lin T{T}K{K}")
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=N)), fmt)
    y32 = S.sharq_linear(a, wq, dtype=torch.float32)
    y16 = S.sharq_linear(a, wq, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    wo = G.weight_to_oracle(wq)
    gemm_check(G.host(y32), O.linear(o, wo), O.linear_abs(o, wo), f"{fmt} T{T}N{N}K{K}")
    assert torch.equal(y16, y32.to(torch.bfloat16))


def test_pairs_llama_qkv_nvfp4_sampled(S, G):
    """The paper's setting (NVFP4, 4:8 in pairs) at the Llama-3.1-8B QKV shape,
    M = 2048: preparation in full, the GEMM on 256 sampled rows x all columns."""
    K, N, _ = synth.LLAMA_LINEARS["qkv"]
    T = 2048
    x = synth.activations(T, K, seed=0)
    a, o = check_prep_pairs(S, G, x, synth.gamma(K, seed=0), synth.LLAMA_EPS, "nv", "llama-qkv")
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=0)), "nv")
    y = S.sharq_linear(a, wq, dtype=torch.float32)
    torch.cuda.synchronize()
    rows = np.random.default_rng(0).choice(T, 256, replace=False)
    rows.sort()
    wo = G.weight_to_oracle(wq)
    gemm_check(G.host(y)[rows], O.linear(o, wo, rows), O.linear_abs(o, wo, rows), "nv llama qkv")
