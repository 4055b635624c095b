"""Path combinations (Sec. 4.4, table "ablation-combination") on the HIP path,
through the C ABI, against the CPU oracle.

Preparation must match the oracle byte for byte in every mode (codes,
metadata and scales of both paths, the NVFP4 per-tensor scale as fp32 bits);
the GEMM must meet the 1e-3 accumulation gate of the method's own GEMM.
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
MODES = ["sparse", "dense", "dense_dense", "sparse_sparse"]


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


def check_prep(S, G, x, g, eps, n, m, fmt, mode, pairs, tag):
    say(f"[mode-prep] {tag} {mode} {fmt} shape={x.shape} {n}:{m}{'p' if pairs else ''} gamma={g is not None}")
    xd = G.dev_bf16(x)
    gd = None if g is None else G.dev_bf16(g)
    a = S.sharq_prepare(xd, gd, eps, n, m, fmt, pairs=pairs, mode=mode)
    torch.cuda.synchronize()
    o = O.prepare_mode(x, g, eps, n, m, fmt, mode, pairs=pairs)
    if fmt == "nv":
        got = np.asarray(G.host(a.tensor_scale)[0], np.float32).view(np.uint32)
        assert got == np.asarray(o["tensor_scale"], np.float32).view(np.uint32), tag
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS_ALL:
        t = a.dn_meta if name == "dn_meta" else getattr(a, name)
        G.assert_bytes_equal(f"{tag}:{mode}:{name}", G.host(t), dev[name])
    return a, o


PREP_CASES = [
    # (T, K, gamma, n, m, pairs, fmt)
    (8, 128, True, 2, 4, False, "mx"),
    (37, 416, True, 2, 4, False, "mx"),
    (37, 416, False, 4, 8, False, "mx"),
    (19, 640, True, 4, 8, True, "mx"),
    (64, 4096, True, 2, 4, False, "mx"),
    (5, 16384, True, 4, 8, False, "mx"),
    (9, 14336, False, 2, 4, False, "mx"),
    (8, 128, True, 2, 4, False, "nv"),
    (37, 416, False, 2, 4, False, "nv"),
    (23, 1024, True, 4, 8, True, "nv"),
    (33, 3584, True, 4, 8, False, "nv"),
    (4, 18944, False, 2, 4, False, "nv"),
]


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("T,K,use_gamma,n,m,pairs,fmt", PREP_CASES)
def test_mode_prep_bit_exact(S, G, mode, T, K, use_gamma, n, m, pairs, fmt):
    x = synth.activations(T, K, seed=T + K)
    g = synth.gamma(K, seed=K) if use_gamma else None
    check_prep(S, G, x, g, 1e-6, n, m, fmt, mode, pairs, f"T{T}K{K}")


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_mode_prep_edge_values(S, G, mode, fmt):
    """All-zero rows, exact ties and tiny blocks next to saturating ones."""
    T, K = 12, 256
    rng = np.random.default_rng(7)
    x = rng.integers(-3, 4, size=(T, K)).astype(np.float32)
    x[0] = 0.0
    x[1, ::3] = -0.0
    x[2, ::2] = 1e-30
    x[3] *= 1e6
    x[4, 5::7] = 6000.0
    check_prep(S, G, synth.f32_to_bf16_bits(x), None, 1e-6, 2, 4, fmt, mode, False, "edge")


def gemm_check(y_gpu, y_ref, y_abs, tag):
    gate = O.gemm_gate_error(y_gpu, y_ref, y_abs)
    norm = float(np.abs(y_gpu.astype(np.float64) - y_ref).max() / max(np.abs(y_ref).max(), 1e-300))
    say(f"[mode-gemm] {tag}: gate={gate:.3e} normwise={norm:.3e}")
    assert gate <= GATE, (tag, gate)
    assert norm <= GATE, (tag, norm)


LINEAR_CASES = [
    # (T, N, K, n, m, pairs)
    (8, 64, 128, 2, 4, False),
    (300, 200, 416, 2, 4, False),
    (129, 300, 640, 4, 8, False),
    (256, 512, 2048, 4, 8, True),
    (1, 256, 3584, 2, 4, False),
]


@pytest.mark.parametrize("fmt", ["mx", "nv"])
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("T,N,K,n,m,pairs", LINEAR_CASES)
def test_mode_linear_parity(S, G, fmt, mode, T, N, K, n, m, pairs):
    """The GEMM on oracle-prepared operands, every output dtype."""
    say(f"[mode-linear] {mode} {fmt} T={T} N={N} K={K} {n}:{m}{'p' if pairs else ''}")
    x = synth.activations(T, K, seed=T + 5)
    o = O.prepare_mode(x, synth.gamma(K, seed=3), 1e-6, n, m, fmt, mode, pairs=pairs)
    wo = O.quantize_weight(synth.weight(N, K, seed=N + 7), fmt)
    a, w = G.oracle_to_act(o), G.oracle_to_weight(wo)
    y32 = S.sharq_linear(a, w, dtype=torch.float32)
    y16 = S.sharq_linear(a, w, dtype=torch.bfloat16)
    yh = S.sharq_linear(a, w, dtype=torch.float16)
    torch.cuda.synchronize()
    gemm_check(G.host(y32), O.linear(o, wo), O.linear_abs(o, wo), f"{mode}-{fmt}-T{T}N{N}K{K}")
    assert torch.equal(y16, y32.to(torch.bfloat16))
    if fmt == "mx":
        assert torch.equal(yh, y32.to(torch.float16))
    else:
        # NVFP4 applies S_x S_w to the fp32 sums; the f16 store may round that
        # exact product once instead of after its fp32 rounding: 1 ulp apart
        ulp = torch.finfo(torch.float16).eps * y32.abs() + 2.0 ** -24
        assert torch.all((yh.float() - y32).abs() <= ulp)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
@pytest.mark.parametrize("mode", MODES)
def test_mode_end_to_end_on_device(S, G, fmt, mode):
    """Prep + weight quantization + GEMM all on the device, against the oracle
    run on the same inputs; the device buffers are also decoded and compared."""
    T, N, K = 96, 320, 1024
    x, g, w = synth.activations(T, K, seed=21), synth.gamma(K, seed=21), synth.weight(N, K, seed=21)
    a, o = check_prep(S, G, x, g, 1e-6, 2, 4, fmt, mode, False, "e2e")
    wq = S.sharq_quantize_weight(G.dev_bf16(w), fmt)
    y = S.sharq_linear(a, wq, dtype=torch.float32)
    torch.cuda.synchronize()
    wo = O.quantize_weight(w, fmt)
    back = G.act_to_oracle(a)
    gemm_check(G.host(y), O.linear(back, wo), O.linear_abs(back, wo), f"e2e-{mode}-{fmt}")


@pytest.mark.parametrize("mode", MODES)
def test_mode_empty(S, G, mode):
    x = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    a = S.sharq_prepare(x, None, 1e-6, 2, 4, "mx", mode=mode)
    w = S.sharq_quantize_weight(G.dev_bf16(synth.weight(64, 256, seed=1)))
    y = S.sharq_linear(a, w)
    torch.cuda.synchronize()
    assert a.rows == 0 and y.shape == (0, 64)


LLAMA_T = 2048


@pytest.mark.parametrize("mode", MODES)
def test_mode_llama_qkv_full_shape(S, G, mode):
    """Full M = 2048 Llama-3.1-8B qkv shape (K 4096, N 6144, MXFP4 2:4):
    preparation compared in full, the GEMM on 256 sampled rows x all columns, and every output written."""
    K, N, _ = synth.LLAMA_LINEARS["qkv"]
    x, g = synth.activations(LLAMA_T, K, seed=1), synth.gamma(K, seed=1)
    a, o = check_prep(S, G, x, g, synth.LLAMA_EPS, 2, 4, "mx", mode, False, "qkv")
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=1)))
    y = torch.full((LLAMA_T, N), float("nan"), dtype=torch.float32, device="cuda")
    S.sharq_linear(a, wq, out=y)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all()), "outputs left unwritten"
    wo = G.weight_to_oracle(wq)
    rows = np.random.default_rng(2).choice(LLAMA_T, 256, replace=False)
    rows[0], rows[1] = 0, LLAMA_T - 1
    gemm_check(G.host(y)[rows], O.linear(o, wo, rows=rows), O.linear_abs(o, wo, rows=rows), f"qkv-{mode}")


def mode_exact_operands(T, N, K, n, m, fmt, mode, seed):
    """Operands of a path combination built directly from random codes (every
    code) under unit block scales (E8M0 127, or E4M3 1.0 with unit per-tensor
    scales): every product is a multiple of 1/4 below 36 and 2 K 36 < 2^22, so
    every fp32 partial sum is exact whatever the order."""
    rng = np.random.default_rng(seed)
    one = 127 if fmt == "mx" else 0x38

    def codes(shape):
        return rng.integers(0, 16, size=shape).astype(np.uint8)

    def path(kind):
        if kind is None:
            z = np.zeros((T, 0), np.uint8)
            return z, z, z
        if kind == "dense":
            return O.pack_nibbles(codes((T, K))), np.zeros((T, 0), np.uint8), \
                np.full((T, K // (32 if fmt == "mx" else 16)), one, np.uint8)
        keep = np.zeros((T, K // m, m), bool)
        np.put_along_axis(keep, rng.random((T, K // m, m)).argsort(axis=2)[..., :n], True, axis=2)
        keep = keep.reshape(T, K)
        c, meta = O.pack_backbone(np.where(keep, codes((T, K)), 0).astype(np.uint8), keep, n, m)
        return c, meta, np.full((T, K // 32), one, np.uint8)

    k1, k2 = O.MODE_PATHS[mode]
    c1, m1, s1 = path(k1)
    c2, m2, s2 = path(k2)
    act = {"rows": T, "K": K, "n": n, "m": m, "pairs": False, "fmt": fmt, "mode": mode,
           "tensor_scale": None if fmt == "mx" else np.float32(1.0),
           "sp_codes": c1, "sp_meta": m1, "sp_scale": s1, "dn_codes": c2, "dn_meta": m2, "dn_scale": s2}
    ws = np.full((N, K // 32), one, np.uint8)
    wq = {"N": N, "K": K, "fmt": fmt, "codes": O.pack_nibbles(codes((N, K))), "scale": ws,
          "scale_dn": ws if fmt == "mx" else np.repeat(ws, 2, axis=1),
          "tensor_scale": None if fmt == "mx" else np.float32(1.0)}
    return act, wq


@pytest.mark.parametrize("fmt", ["mx", "nv"])
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("T,N,K,n,m", [(300, 520, 1024, 2, 4), (130, 300, 416, 4, 8)])
def test_mode_exact_sums(S, G, fmt, mode, T, N, K, n, m):
    """Every path combination's GEMM on exact-sum operands equals the
    oracle's exact result bit for bit."""
    say(f"[mode-exact] {mode} {fmt} T={T} N={N} K={K} {n}:{m}")
    o, wo = mode_exact_operands(T, N, K, n, m, fmt, mode, seed=T + K + len(mode))
    y = S.sharq_linear(G.oracle_to_act(o), G.oracle_to_weight(wo), dtype=torch.float32)
    torch.cuda.synchronize()
    ref = O.linear(o, wo)
    got = G.host(y).astype(np.float64)
    bad = np.nonzero(got != ref)
    assert bad[0].size == 0, (f"{mode} {fmt}: {bad[0].size} outputs differ from the exact sum; first at "
                              f"{bad[0][0]},{bad[1][0]}: {got[bad[0][0], bad[1][0]]} vs {ref[bad[0][0], bad[1][0]]}")
