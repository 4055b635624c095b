"""HiF4 on the HIP path (App. "HiFloat4 (HiF4) Data Format"; the paper pairs
it with the 2:4 backbone), through the C ABI, against the CPU oracle:
preparation and weight quantization byte for byte, the GEMM (bf16 MFMA over
exactly dequantized operands) within the 1e-3 accumulation gate."""

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


def check_prep(S, G, x, g, eps, tag):
    say(f"[hif4-prep] {tag} shape={x.shape} gamma={g is not None}")
    a = S.sharq_prepare(G.dev_bf16(x), None if g is None else G.dev_bf16(g), eps, 2, 4, "hif4")
    torch.cuda.synchronize()
    o = O.prepare(x, g, eps, 2, 4, "hif4")
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(f"{tag}:{name}", G.host(getattr(a, name)), dev[name])
    return a, o


@pytest.mark.parametrize("T,K,use_gamma", [(8, 128, True), (37, 448, True), (37, 448, False), (64, 4096, True),
                                           (5, 16384, True), (9, 14336, False), (3, 64, False)])
def test_hif4_prep_bit_exact(S, G, T, K, use_gamma):
    x = synth.activations(T, K, seed=T + K)
    check_prep(S, G, x, synth.gamma(K, seed=K) if use_gamma else None, 1e-6, f"T{T}K{K}")


@pytest.mark.parametrize("kind", ["zeros", "ties", "huge", "tiny", "mixed"])
def test_hif4_prep_edge_values(S, G, kind):
    T, K = 12, 256
    rng = np.random.default_rng(len(kind))
    if kind == "zeros":
        x = np.zeros((T, K), np.float32)
        x[:, ::3] = -0.0
    elif kind == "ties":
        x = rng.integers(-3, 4, size=(T, K)).astype(np.float32)
    elif kind == "huge":                  # level-1 scales clamped at 1.5 * 2^15
        x = (rng.standard_normal((T, K)) * 1e30).astype(np.float32)
    elif kind == "tiny":                  # below the smallest level-1 scale
        x = (rng.standard_normal((T, K)) * 1e-20).astype(np.float32)
    else:
        x = rng.standard_normal((T, K)).astype(np.float32)
        x[0] = 0.0
        x[1, ::2] = 1e-30
        x[2] *= 1e6
        x[3, 5::7] = 6000.0
    check_prep(S, G, synth.f32_to_bf16_bits(x), None, 1e-6, f"hif4-edge-{kind}")


@pytest.mark.parametrize("N,K,dt", [(64, 128, "bf16"), (200, 448, "bf16"), (4096, 4096, "bf16"), (33, 14336, "bf16"),
                                    (96, 256, "f32")])
def test_hif4_weight_quant_bit_exact(S, G, N, K, dt):
    say(f"[hif4-wquant] N={N} K={K} {dt}")
    w = synth.weight(N, K, seed=N + 1)
    wd = G.dev_bf16(w) if dt == "bf16" else torch.from_numpy(O.bf16_bits_to_f32(w)).cuda()
    q = S.sharq_quantize_weight(wd, "hif4")
    torch.cuda.synchronize()
    o = L.weight_to_device_layout(O.quantize_weight(w, "hif4"))
    G.assert_bytes_equal("codes", G.host(q.codes[0]), o["codes"])
    G.assert_bytes_equal("scale", G.host(q.scale[0]), o["scale"])


def gemm_check(y_gpu, y_ref, y_abs, tag):
    gate = O.gemm_gate_error(y_gpu, y_ref, y_abs)
    norm = float(np.abs(y_gpu.astype(np.float64) - y_ref).max() / max(np.abs(y_ref).max(), 1e-300))
    say(f"[hif4-gemm] {tag}: gate={gate:.3e} normwise={norm:.3e}")
    assert gate <= GATE, (tag, gate)
    assert norm <= GATE, (tag, norm)


@pytest.mark.parametrize("T,N,K", [(8, 64, 128), (300, 200, 448), (1, 256, 3584), (129, 300, 640), (256, 512, 2048),
                                   (16, 4096, 14336)])
def test_hif4_linear_parity(S, G, T, N, K):
    say(f"[hif4-linear] T={T} N={N} K={K}")
    x = synth.activations(T, K, seed=T + 5)
    o = O.prepare(x, synth.gamma(K, seed=3), 1e-6, 2, 4, "hif4")
    wo = O.quantize_weight(synth.weight(N, K, seed=N + 7), "hif4")
    a, w = G.oracle_to_act(o), G.oracle_to_weight(wo)
    y32 = S.sharq_linear(a, w, dtype=torch.float32)
    y16 = S.sharq_linear(a, w, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    gemm_check(G.host(y32), O.linear(o, wo), O.linear_abs(o, wo), f"T{T}N{N}K{K}")
    assert torch.equal(y16, y32.to(torch.bfloat16))


def test_hif4_end_to_end_on_device(S, G):
    T, N, K = 96, 320, 1024
    x, g, w = synth.activations(T, K, seed=21), synth.gamma(K, seed=21), synth.weight(N, K, seed=21)
    a, o = check_prep(S, G, x, g, 1e-6, "e2e")
    wq = S.sharq_quantize_weight(G.dev_bf16(w), "hif4")
    y = S.sharq_linear(a, wq, dtype=torch.float32)
    torch.cuda.synchronize()
    wo = O.quantize_weight(w, "hif4")
    gemm_check(G.host(y), O.linear(o, wo), O.linear_abs(o, wo), "e2e")


def test_hif4_empty(S, G):
    a = S.sharq_prepare(torch.empty((0, 256), dtype=torch.bfloat16, device="cuda"), None, 1e-6, 2, 4, "hif4")
    w = S.sharq_quantize_weight(G.dev_bf16(synth.weight(64, 256, seed=1)), "hif4")
    y = S.sharq_linear(a, w)
    torch.cuda.synchronize()
    assert a.rows == 0 and y.shape == (0, 64)


@pytest.mark.parametrize("name", ["qkv", "down"])
def test_hif4_llama_full_shape(S, G, name):
    """Full M = 2048 Llama-3.1-8B shapes: preparation compared in full, the
    GEMM on 256 sampled rows x all columns, and every output written."""
    K, N, norm = synth.LLAMA_LINEARS[name]
    x = synth.activations(2048, K, seed=1)
    a, o = check_prep(S, G, x, synth.gamma(K, seed=1) if norm else None, synth.LLAMA_EPS, name)
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=1)), "hif4")
    y = torch.full((2048, N), float("nan"), dtype=torch.float32, device="cuda")
    S.sharq_linear(a, wq, out=y)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all()), "outputs left unwritten"
    wo = G.weight_to_oracle(wq)
    rows = np.random.default_rng(2).choice(2048, 256, replace=False)
    rows[0], rows[1] = 0, 2048 - 1
    gemm_check(G.host(y)[rows], O.linear(o, wo, rows=rows), O.linear_abs(o, wo, rows=rows), name)


def hif4_exact_operands(T, N, K, seed):
    """A HiF4 prepared activation (2:4) and weight built directly from codes
    and unit metadata: activation units with E6M2 scales in {1/2, 1, 2},
    weight units with every mantissa, {1, 1.25, 1.5, 1.75}, and random
    micro-exponent bits on both sides.  Every activation value is a multiple of
    1/8 and every weight value of 1/16, so every product is a multiple of
    1/128; the S1P2 magnitudes are limited so that the at most 2K products of
    an output, each below max|a| max|w|, stay below 2^24 / 128: every fp32
    partial sum is then exact whatever the order."""
    rng = np.random.default_rng(seed)
    ma, mw = 7, 7
    while 2 * K * (ma / 4 * 4 * 2) * (mw / 4 * 4 * 1.75) * 128 >= 2.0 ** 24:
        if ma >= mw:
            ma -= 1
        else:
            mw -= 1
    keep = np.zeros((T, K // 4, 4), bool)
    order = rng.random((T, K // 4, 4)).argsort(axis=2)[..., :2]
    np.put_along_axis(keep, order, True, axis=2)
    keep = keep.reshape(T, K)

    def codes(shape, mmax):
        return (rng.integers(0, mmax + 1, size=shape) | (rng.integers(0, 2, size=shape) << 3)).astype(np.uint8)

    def meta(rows, bases):
        U = K // 64
        m = np.zeros((rows, U, 4), np.uint8)
        m[..., 0] = np.asarray(bases, np.uint8)[rng.integers(0, len(bases), size=(rows, U))]
        m[..., 1:] = rng.integers(0, 256, size=(rows, U, 3))
        return m.reshape(rows, U * 4)

    act_bases, w_bases = [47 * 4, 48 * 4, 49 * 4], [48 * 4, 48 * 4 + 1, 48 * 4 + 2, 48 * 4 + 3]
    sp = np.where(keep, codes((T, K), ma), 0).astype(np.uint8)
    sp_codes, sp_meta = O.pack_backbone(sp, keep, 2, 4)
    act = {"rows": T, "K": K, "n": 2, "m": 4, "pairs": False, "fmt": "hif4", "tensor_scale": None, "mode": "sharq",
           "sp_codes": sp_codes, "sp_meta": sp_meta, "sp_scale": meta(T, act_bases),
           "dn_codes": O.pack_nibbles(codes((T, K), ma)), "dn_scale": meta(T, act_bases),
           "dn_meta": np.zeros((T, 0), np.uint8)}
    wm = meta(N, w_bases)
    wq = {"N": N, "K": K, "fmt": "hif4", "codes": O.pack_nibbles(codes((N, K), mw)), "scale": wm, "scale_dn": wm,
          "tensor_scale": None}
    return act, wq, (ma, mw)


@pytest.mark.parametrize("T,N,K", [(300, 520, 1024), (130, 300, 448), (2048, 4096, 4096)])
def test_hif4_exact_sums(S, G, T, N, K):
    """The HiF4 GEMM on operands whose sums are exact in fp32: the output
    equals the oracle's exact result bit for bit (all rows, or 256 sampled at
    M = 2048), so a dropped or repeated product or a misread micro-exponent,
    E6M2 mantissa or unit shows."""
    o, wo, mags = hif4_exact_operands(T, N, K, seed=T + N + K)
    say(f"[hif4-exact] T={T} N={N} K={K} code magnitude limits {mags}")
    y = S.sharq_linear(G.oracle_to_act(o), G.oracle_to_weight(wo), dtype=torch.float32)
    torch.cuda.synchronize()
    rows = np.arange(T) if T <= 512 else np.random.default_rng(7).choice(T, 256, replace=False)
    ref = O.linear(o, wo, rows=rows)
    got = G.host(y)[rows].astype(np.float64)
    bad = np.nonzero(got != ref)
    assert bad[0].size == 0, (f"{bad[0].size} outputs differ from the exact sum; first at {bad[0][0]},{bad[1][0]}: "
                              f"{got[bad[0][0], bad[1][0]]} vs {ref[bad[0][0], bad[1][0]]}")
