"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Preparation and weight quantization must match the oracle byte for byte; the
two-path GEMM must match the oracle's fp64 result within the componentwise
accumulation gate max|Y^ - Y| / sum_k(|a_sp w| + |a_dn w|) <= 1e-3 and the
normwise bound max|Y^ - Y| / max|Y| <= 1e-3.
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


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def special_rows(kind: str, T: int, K: int, seed: int) -> np.ndarray:
    """Edge-case activations (bf16 bits)."""
    rng = np.random.default_rng(seed)
    if kind == "zeros":
        x = np.zeros((T, K), np.float32)
        x[:, ::3] = -0.0
    elif kind == "ties":
        x = rng.integers(-3, 4, size=(T, K)).astype(np.float32)
    elif kind == "subnormal":
        x = (rng.standard_normal((T, K)) * 1e-39).astype(np.float32)
        x[:, ::5] *= 1e-2
    elif kind == "huge":
        x = (rng.standard_normal((T, K)) * 1e30).astype(np.float32)
    elif kind == "mixed":
        x = rng.standard_normal((T, K)).astype(np.float32)
        x[0] = 0.0
        x[1, ::2] = 1e-40
        x[2] *= 1e25
        x[3, 5::7] = 6000.0
    else:
        raise ValueError(kind)
    return synth.f32_to_bf16_bits(x)


def run_prep(S, G, x_u16, gamma_u16, eps, n, m):
    x = G.dev_bf16(x_u16)
    g = None if gamma_u16 is None else G.dev_bf16(gamma_u16)
    a = S.sharq_prepare(x, g, eps, n, m, "mx")
    torch.cuda.synchronize()
    return a


def check_prep(S, G, x_u16, gamma_u16, eps, n, m, tag):
    say(f"[prep] {tag} shape={x_u16.shape} n:m={n}:{m} gamma={gamma_u16 is not None}")
    a = run_prep(S, G, x_u16, gamma_u16, eps, n, m)
    o = O.prepare(x_u16, gamma_u16, eps, n, m, "mx")
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(f"{tag}:{name}", G.host(getattr(a, name)), dev[name])
    return a, o


@pytest.fixture(scope="module")
def G(S):
    import gpu_util
    return gpu_util


PREP_CASES = [
    # (T, K, gamma, n, m, eps)
    (8, 128, True, 2, 4, 1e-6),
    (37, 416, True, 2, 4, 1e-5),
    (37, 416, False, 2, 4, 1e-5),
    (37, 416, True, 4, 8, 1e-5),
    (3, 32, True, 2, 4, 1e-6),
    (64, 4096, True, 2, 4, 1e-5),
    (17, 3584, True, 2, 4, 1e-6),
    (9, 16384, True, 2, 4, 1e-5),
    (5, 14336, False, 2, 4, 1e-5),
    (130, 2048, True, 4, 8, 1e-6),
    (33, 768, False, 4, 8, 1e-6),
    (6, 18944, False, 2, 4, 1e-6),
]


@pytest.mark.parametrize("T,K,use_gamma,n,m,eps", PREP_CASES)
def test_prep_bit_exact(S, G, T, K, use_gamma, n, m, eps):
    x = synth.activations(T, K, seed=T + K)
    g = synth.gamma(K, seed=K) if use_gamma else None
    check_prep(S, G, x, g, eps, n, m, f"T{T}K{K}")


@pytest.mark.parametrize("kind", ["zeros", "ties", "subnormal", "huge", "mixed"])
@pytest.mark.parametrize("use_gamma", [True, False])
@pytest.mark.parametrize("n,m", [(2, 4), (4, 8)])
def test_prep_edge_values(S, G, kind, use_gamma, n, m):
    T, K = 12, 256
    x = special_rows(kind, T, K, seed=len(kind))
    g = synth.gamma(K, seed=3) if use_gamma else None
    if kind == "zeros" and use_gamma:
        g = synth.gamma(K, seed=3)   # all-zero rows: r = 1/sqrt(eps), y = 0
    check_prep(S, G, x, g, 1e-6, n, m, f"edge-{kind}")


def test_prep_empty(S, G):
    x = torch.empty((0, 128), dtype=torch.bfloat16, device="cuda")
    a = S.sharq_prepare(x, None, 1e-6, 2, 4, "mx")
    torch.cuda.synchronize()
    assert a.rows == 0 and a.dn_codes.numel() == 0


def test_prep_strided_rows(S, G):
    """A row stride larger than K (ldx > K) reads only the first K columns."""
    T, K, ld = 20, 256, 384
    full = synth.activations(T, ld, seed=7)
    xd = G.dev_bf16(full)[:, :K]
    a = S.sharq_prepare(xd, None, 1e-6, 2, 4, "mx")
    torch.cuda.synchronize()
    o = O.prepare(np.ascontiguousarray(full[:, :K]), None, 1e-6, 2, 4, "mx")
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(name, G.host(getattr(a, name)), dev[name])


@pytest.mark.parametrize("N,K", [(64, 128), (200, 416), (6144, 4096), (33, 14336)])
def test_weight_quant_bit_exact(S, G, N, K):
    say(f"[wquant] N={N} K={K}")
    w = synth.weight(N, K, seed=N)
    q = S.sharq_quantize_weight(G.dev_bf16(w), "mx")
    torch.cuda.synchronize()
    o = L.weight_to_device_layout(O.quantize_weight(w, "mx"))
    G.assert_bytes_equal("codes", G.host(q.codes[0]), o["codes"])
    G.assert_bytes_equal("scale", G.host(q.scale[0]), o["scale"])


def test_weight_quant_fp32_input(S, G):
    w = synth.weight(96, 256, seed=5)
    wf = torch.from_numpy(O.bf16_bits_to_f32(w)).cuda()
    q = S.sharq_quantize_weight(wf, "mx")
    torch.cuda.synchronize()
    o = L.weight_to_device_layout(O.quantize_weight(w, "mx"))
    G.assert_bytes_equal("codes", G.host(q.codes[0]), o["codes"])


def gemm_check(y_gpu: np.ndarray, y_ref: np.ndarray, y_abs: np.ndarray, tag: str):
    gate = O.gemm_gate_error(y_gpu, y_ref, y_abs)
    norm = float(np.abs(y_gpu.astype(np.float64) - y_ref).max() / max(np.abs(y_ref).max(), 1e-300))
    say(f"[gemm] {tag}: gate={gate:.3e} normwise={norm:.3e}")
    assert gate <= GATE, (tag, gate)
    assert norm <= GATE, (tag, norm)


LINEAR_CASES = [
    # (T, N, K, n, m)
    (8, 64, 128, 2, 4),
    (300, 200, 416, 2, 4),
    (1, 256, 4096, 2, 4),
    (129, 300, 640, 4, 8),
    (256, 512, 2048, 2, 4),
    (16, 6144, 4096, 2, 4),
]


@pytest.mark.parametrize("T,N,K,n,m", LINEAR_CASES)
def test_linear_parity(S, G, T, N, K, n, m):
    say(f"[linear] T={T} N={N} K={K} {n}:{m}")
    x = synth.activations(T, K, seed=T)
    o = O.prepare(x, synth.gamma(K, seed=1), 1e-6, n, m, "mx")
    wo = O.quantize_weight(synth.weight(N, K, seed=N), "mx")
    a = G.oracle_to_act(o)
    w = G.oracle_to_weight(wo)
    y32 = S.sharq_linear(a, w, dtype=torch.float32)
    y16 = S.sharq_linear(a, w, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    ref = O.linear(o, wo)
    gemm_check(G.host(y32), ref, O.linear_abs(o, wo), f"T{T}N{N}K{K}")
    # bf16 output is the fp32 result rounded once
    assert torch.equal(y16, y32.to(torch.bfloat16))


def test_linear_ldy_and_empty(S, G):
    T, N, K = 40, 96, 256
    x = synth.activations(T, K, seed=2)
    o = O.prepare(x, None, 1e-6, 2, 4, "mx")
    wo = O.quantize_weight(synth.weight(N, K, seed=2), "mx")
    a, w = G.oracle_to_act(o), G.oracle_to_weight(wo)
    big = torch.full((T, 128), 7.0, dtype=torch.float32, device="cuda")
    S.sharq_linear(a, w, out=big[:, :N])
    torch.cuda.synchronize()
    assert torch.all(big[:, N:] == 7.0)
    gemm_check(G.host(big[:, :N]), O.linear(o, wo), O.linear_abs(o, wo), "ldy")
    e = S.sharq_prepare(torch.empty((0, K), dtype=torch.bfloat16, device="cuda"), None, 1e-6, 2, 4)
    y = S.sharq_linear(e, w, dtype=torch.float32)
    torch.cuda.synchronize()
    assert y.shape == (0, N)


def test_end_to_end_deterministic(S, G):
    T, N, K = 96, 320, 1024
    x = G.dev_bf16(synth.activations(T, K, seed=4))
    g = G.dev_bf16(synth.gamma(K, seed=4))
    w = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=4)))
    outs = []
    for _ in range(2):
        a = S.sharq_prepare(x, g, 1e-5, 2, 4)
        outs.append(S.sharq_linear(a, w, dtype=torch.float32))
    torch.cuda.synchronize()
    assert torch.equal(outs[0], outs[1])


# --------------------------------------------------------------------------- full Llama shapes

LLAMA_T = 2048


# rows of the full-shape GEMM comparison: every row of qkv and down, 512 of
# gate_up's 2048 (token 0, the massive-activation row, among them)
FULL_ROWS = {"qkv": None, "gate_up": 512, "down": None}


def full_rows(name):
    if FULL_ROWS[name] is None:
        return np.arange(LLAMA_T)
    rows = np.random.default_rng(1).choice(LLAMA_T, FULL_ROWS[name], replace=False)
    rows[0] = 0
    return np.sort(rows)


@pytest.mark.parametrize("name", ["qkv", "gate_up", "down"])
def test_llama_full_shape(S, G, name):
    """Full M=2048 Llama-3.1-8B shapes in the benchmark's launch configuration
    (the preparation writes the dense backbone copy, the GEMM reads it):
    preparation compared in full, dense copy included; the GEMM on every row
    (qkv, down) or 512 rows (gate_up) x all columns against the oracle, and
    bit-identical to the GEMM that expands the compressed backbone."""
    K, N, norm = synth.LLAMA_LINEARS[name]
    say(f"[llama] {name} T={LLAMA_T} K={K} N={N} (dense backbone copy)")
    x = synth.activations(LLAMA_T, K, seed=0)
    g = synth.gamma(K, seed=0) if norm else None
    w = synth.weight(N, K, seed=0)
    xd, gd = G.dev_bf16(x), (None if g is None else G.dev_bf16(g))
    a = S.sharq_prepare(xd, gd, synth.LLAMA_EPS, 2, 4, "mx",
                        out=S.alloc_act(LLAMA_T, K, 2, 4, "mx", "cuda", dense_backbone=True))
    wq = S.sharq_quantize_weight(G.dev_bf16(w))
    y = S.sharq_linear(a, wq, dtype=torch.float32)
    y16 = S.sharq_linear(a, wq, dtype=torch.bfloat16)
    c = S.sharq_prepare(xd, gd, synth.LLAMA_EPS, 2, 4, "mx")
    yc = S.sharq_linear(c, wq, dtype=torch.float32)
    torch.cuda.synchronize()
    o = O.prepare(x, g, synth.LLAMA_EPS, 2, 4, "mx")
    dev = L.act_to_device_layout(o)
    for buf in O.ACT_BUFFERS:
        G.assert_bytes_equal(f"{name}:{buf}", G.host(getattr(a, buf)), dev[buf])
    G.assert_bytes_equal(f"{name}:sp_dense", G.host(a.sp_dense), L.dense_backbone_to_device_layout(o))
    assert torch.equal(y, yc)
    assert torch.equal(y16, y.to(torch.bfloat16))
    wo = G.weight_to_oracle(wq)
    rows = full_rows(name)
    gemm_check(G.host(y)[rows], O.linear(o, wo, rows=rows), O.linear_abs(o, wo, rows=rows), name)


# --------------------------------------------------------------------------- exact sums at full K

def exact_operands(T, N, K, variant, seed):
    """A prepared activation (2:4) and a weight built directly from random
    codes and scales such that every fp32 partial sum of the two-path GEMM is
    exact, whatever the order of accumulation:
      'unit'    every E8M0 scale 127 (2^0), all 16 codes: products are
                multiples of 1/4 below 36, and 2 K 36 < 2^22 for K <= 14336;
      'act'     activation scales in {126, 127, 128} with activation codes of
                magnitude <= 2, weight scales 127: multiples of 1/8 below 24;
      'weight'  the same with the roles exchanged.
    The fp32 result must then equal the exact (fp64) sum bit for bit, so a
    single dropped, repeated or misplaced product shows."""
    rng = np.random.default_rng(seed)
    pairs = np.array([(0, 1), (0, 2), (0, 3), (1, 2), (1, 3), (2, 3)])
    sel = pairs[rng.integers(0, 6, size=(T, K // 4))]
    keep = np.zeros((T, K // 4, 4), bool)
    t, gi = np.meshgrid(np.arange(T), np.arange(K // 4), indexing="ij")
    keep[t, gi, sel[..., 0]] = True
    keep[t, gi, sel[..., 1]] = True
    keep = keep.reshape(T, K)

    def codes(shape, small):
        mag = rng.integers(0, 5 if small else 8, size=shape)
        return (mag | (rng.integers(0, 2, size=shape) << 3)).astype(np.uint8)

    def scales(shape, vary):
        return (rng.integers(126, 129, size=shape) if vary else np.full(shape, 127)).astype(np.uint8)

    small_a, small_w = variant == "act", variant == "weight"
    sp = np.where(keep, codes((T, K), small_a), 0).astype(np.uint8)
    sp_codes, sp_meta = O.pack_backbone(sp, keep, 2, 4)
    act = {"rows": T, "K": K, "n": 2, "m": 4, "pairs": False, "fmt": "mx", "tensor_scale": None, "mode": "sharq",
           "sp_codes": sp_codes, "sp_meta": sp_meta, "sp_scale": scales((T, K // 32), small_a),
           "dn_codes": O.pack_nibbles(codes((T, K), small_a)), "dn_scale": scales((T, K // 32), small_a),
           "dn_meta": np.zeros((T, 0), np.uint8)}
    wq = {"N": N, "K": K, "fmt": "mx", "tensor_scale": None, "codes": O.pack_nibbles(codes((N, K), small_w)),
          "scale": scales((N, K // 32), small_w)}
    wq["scale_dn"] = wq["scale"]
    return act, wq


@pytest.mark.parametrize("variant", ["unit", "act", "weight"])
@pytest.mark.parametrize("name", ["qkv", "gate_up", "down"])
def test_exact_sums_full_shape(S, G, name, variant):
    """The benchmarked GEMM (dense backbone copy) and the compressed-backbone
    GEMM at the full Llama shapes, on operands whose sums are exact in fp32:
    the output must equal the oracle's exact result bit for bit (every row of
    qkv and down, 512 rows of gate_up)."""
    K, N, _ = synth.LLAMA_LINEARS[name]
    say(f"[exact] {name} T={LLAMA_T} K={K} N={N} variant={variant}")
    o, wo = exact_operands(LLAMA_T, N, K, variant, seed=K + N + len(variant))
    a = G.oracle_to_act(o, dense_backbone=True)
    w = G.oracle_to_weight(wo)
    yd = S.sharq_linear(a, w, dtype=torch.float32)
    a.sp_dense = None
    yc = S.sharq_linear(a, w, dtype=torch.float32)
    torch.cuda.synchronize()
    rows = full_rows(name)
    ref = O.linear(o, wo, rows=rows)
    for tag, y in (("dense copy", yd), ("compressed", yc)):
        got = G.host(y)[rows].astype(np.float64)
        bad = np.nonzero(got != ref)
        assert bad[0].size == 0, (f"{name} {variant} {tag}: {bad[0].size} outputs differ from the exact sum; "
                                  f"first at {bad[0][0]},{bad[1][0]}: {got[bad[0][0], bad[1][0]]} "
                                  f"vs {ref[bad[0][0], bad[1][0]]}")


@pytest.mark.parametrize("name,T,variant", [("qkv", 1, "unit"), ("gate_up", 4, "act"), ("down", 16, "weight"),
                                            ("gate_up", 32, "unit"), ("down", 64, "act"), ("qkv", 256, "weight")])
def test_exact_sums_decode(S, G, name, T, variant):
    """The small-M kernels (K split over wavefronts, partial tiles added in
    LDS) on exact-sum operands at the Llama shapes: the output equals the
    oracle's exact result bit for bit, on the dense backbone copy and on the
    compressed backbone, so a lost or doubled partial tile shows."""
    K, N, _ = synth.LLAMA_LINEARS[name]
    say(f"[exact-decode] {name} T={T} K={K} N={N} variant={variant}")
    o, wo = exact_operands(T, N, K, variant, seed=K + N + T)
    w = G.oracle_to_weight(wo)
    yd = S.sharq_linear(G.oracle_to_act(o, dense_backbone=True), w, dtype=torch.float32)
    yc = S.sharq_linear(G.oracle_to_act(o), w, dtype=torch.float32)
    torch.cuda.synchronize()
    ref = O.linear(o, wo)
    for tag, y in (("dense copy", yd), ("compressed", yc)):
        got = G.host(y).astype(np.float64)
        bad = np.nonzero(got != ref)
        assert bad[0].size == 0, (f"{name} T={T} {variant} {tag}: {bad[0].size} outputs differ from the exact sum; "
                                  f"first at {bad[0][0]},{bad[1][0]}")


@pytest.mark.parametrize("gather", [True, False])
def test_exact_sums_grouped(S, G, gather):
    """The grouped GEMM on exact-sum operands (unit scales, all codes): with
    a row map (the gathering kernel and its spread load schedule) and on
    expert-sorted rows, on the dense backbone copy and on the compressed
    backbone, the output equals the oracle's exact result bit for bit."""
    T, E, topk, K, N = 512, 16, 4, 2048, 520
    row_index, offs = synth.router_topk(T, E, topk, seed=3)
    total = int(offs[-1])
    rows = T if gather else total
    say(f"[exact-grouped] gather={gather} rows={rows} total={total} E={E} K={K} N={N}")
    o, _ = exact_operands(rows, 32, K, "unit", seed=5)
    wos = [exact_operands(1, N, K, "unit", seed=100 + e)[1] for e in range(E)]
    w = S.stack_weights([G.oracle_to_weight(wo) for wo in wos])
    ri = torch.from_numpy(row_index).cuda() if gather else None
    of = torch.from_numpy(offs).cuda()
    yd = S.sharq_linear_grouped(G.oracle_to_act(o, dense_backbone=True), ri, of, total, w, dtype=torch.float32)
    yc = S.sharq_linear_grouped(G.oracle_to_act(o), ri, of, total, w, dtype=torch.float32)
    torch.cuda.synchronize()
    ref = O.linear_grouped(o, row_index if gather else None, offs, wos)
    for tag, y in (("dense copy", yd), ("compressed", yc)):
        got = G.host(y).astype(np.float64)
        bad = np.nonzero(got != ref)
        assert bad[0].size == 0, (f"gather={gather} {tag}: {bad[0].size} outputs differ from the exact sum; "
                                  f"first at {bad[0][0]},{bad[1][0]}")


# --------------------------------------------------------------------------- decode shapes

@pytest.mark.parametrize("name,T", [("qkv", 1), ("qkv", 16), ("gate_up", 1), ("gate_up", 16), ("gate_up", 32),
                                    ("down", 64), ("gate_up", 33), ("gate_up", 64), ("down", 5), ("qkv", 48),
                                    ("down", 100), ("qkv", 128), ("down", 256)])
def test_llama_decode_shape(S, G, name, T):
    """Small-M (decode) Llama-3.1-8B shapes, as the decode benchmark runs them:
    preparation in full, GEMM on every row."""
    K, N, norm = synth.LLAMA_LINEARS[name]
    say(f"[decode] {name} T={T} K={K} N={N}")
    x = synth.activations(T, K, seed=T)
    g = synth.gamma(K, seed=0) if norm else None
    a, o = check_prep(S, G, x, g, synth.LLAMA_EPS, 2, 4, f"{name}-T{T}")
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=0)))
    y = S.sharq_linear(a, wq, dtype=torch.float32)
    y16 = S.sharq_linear(a, wq, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    wo = G.weight_to_oracle(wq)
    gemm_check(G.host(y), O.linear(o, wo), O.linear_abs(o, wo), f"decode {name} T{T}")
    assert torch.equal(y16, y.to(torch.bfloat16))


@pytest.mark.parametrize("T,N,K,n,m", [(7, 40, 256, 4, 8), (64, 96, 1280, 2, 4), (17, 16, 128, 2, 4),
                                       (70, 40, 256, 2, 4), (200, 96, 1280, 4, 8), (129, 4104, 512, 2, 4),
                                       (3, 12300, 256, 4, 8), (5, 12300, 4096, 2, 4), (11, 6152, 640, 2, 4),
                                       (2, 6200, 16384, 2, 4), (20, 12300, 4096, 4, 8)])
def test_small_m_ragged(S, G, T, N, K, n, m):
    """Small-M kernel: column tails (N % 16), K ranges shorter than four panels,
    4:8, and row tiles with a ragged last tile (M > 64 with few main-kernel tiles).
    At M <= 16 a wide N takes 4 or 2 column fragments per wavefront: N = 12300
    (4 fragments, a 12-column tail; K = 256 leaves two of the four wavefronts
    without a panel, K = 4096 splits K eight ways), N = 6152 (2 fragments, an
    8-column tail) and N = 6200 with K = 16384 (2 fragments, sixteen-way split);
    at M = 20 the same N = 12300 takes 2 row and 4 column fragments."""
    x = synth.activations(T, K, seed=K)
    o = O.prepare(x, synth.gamma(K, seed=2), 1e-6, n, m, "mx")
    wo = O.quantize_weight(synth.weight(N, K, seed=N), "mx")
    a, w = G.oracle_to_act(o), G.oracle_to_weight(wo)
    y = S.sharq_linear(a, w, dtype=torch.float32)
    torch.cuda.synchronize()
    gemm_check(G.host(y), O.linear(o, wo), O.linear_abs(o, wo), f"small-M T{T}N{N}K{K}")


# --------------------------------------------------------------------------- grouped (MoE)

@pytest.mark.parametrize("T,E,topk,K,N", [(64, 8, 2, 256, 96), (300, 5, 3, 416, 200)])
def test_grouped_parity(S, G, T, E, topk, K, N):
    say(f"[grouped] T={T} E={E} top{topk} K={K} N={N}")
    x = synth.activations(T, K, seed=E)
    o = O.prepare(x, synth.gamma(K, seed=E), 1e-6, 4, 8, "mx")
    wos = [O.quantize_weight(synth.weight(N, K, seed=100 + e), "mx") for e in range(E)]
    row_index, offs = synth.router_topk(T, E, topk, seed=E)
    total = int(offs[-1])
    a = G.oracle_to_act(o)
    w = S.stack_weights([G.oracle_to_weight(wo) for wo in wos])
    ri = torch.from_numpy(row_index).cuda()
    of = torch.from_numpy(offs).cuda()
    y = S.sharq_linear_grouped(a, ri, of, total, w, dtype=torch.float32)
    torch.cuda.synchronize()
    ref = O.linear_grouped(o, row_index, offs, wos)
    yabs = np.zeros_like(ref)
    for e in range(E):
        lo, hi = offs[e], offs[e + 1]
        if hi > lo:
            yabs[lo:hi] = O.linear_abs(o, wos[e], rows=row_index[lo:hi])
    gemm_check(G.host(y), ref, yabs, f"grouped T{T}E{E}")


def test_grouped_uneven_experts(S, G):
    """Expert sizes 0, 1, 129, 0, 300 rows; identity row map (row_index = NULL)."""
    K, N = 256, 160
    sizes = [0, 1, 129, 0, 300]
    offs = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    total = int(offs[-1])
    x = synth.activations(total, K, seed=9)
    o = O.prepare(x, None, 1e-6, 2, 4, "mx")
    wos = [O.quantize_weight(synth.weight(N, K, seed=200 + e), "mx") for e in range(len(sizes))]
    a = G.oracle_to_act(o)
    w = S.stack_weights([G.oracle_to_weight(wo) for wo in wos])
    y = S.sharq_linear_grouped(a, None, torch.from_numpy(offs).cuda(), total, w, dtype=torch.float32)
    torch.cuda.synchronize()
    ref = O.linear_grouped(o, None, offs, wos)
    yabs = np.zeros_like(ref)
    for e in range(len(sizes)):
        lo, hi = offs[e], offs[e + 1]
        if hi > lo:
            yabs[lo:hi] = O.linear_abs(o, wos[e], rows=np.arange(lo, hi))
    gemm_check(G.host(y), ref, yabs, "grouped-uneven")


def test_moe_full_config(S, G):
    """Qwen3-30B-A3B expert layers at full size, in the benchmark's launch
    configuration: 4096 tokens, top-8 of 128 experts, gate/up 1536 x 2048 with
    RMSNorm, 4:8.  Preparation compared in full; the grouped GEMM on the
    slices of four experts (all their rows, all columns)."""
    cfg = synth.MOE
    T, H, E, I, k = cfg["tokens"], cfg["hidden"], cfg["experts"], cfg["inter"], cfg["topk"]
    say(f"[moe] T={T} H={H} E={E} I={I} top{k}")
    x = synth.activations(T, H, seed=0)
    g = synth.gamma(H, seed=0)
    a, o = check_prep(S, G, x, g, 1e-6, 4, 8, "moe-gate_up-input")
    ridx, offs = synth.router_topk(T, E, k, seed=0)
    total = int(offs[-1])
    ws = [synth.weight(2 * I, H, seed=100 + e) for e in range(E)]
    w = S.stack_weights([S.sharq_quantize_weight(G.dev_bf16(we)) for we in ws])
    y = S.sharq_linear_grouped(a, torch.from_numpy(ridx).cuda(), torch.from_numpy(offs).cuda(), total, w,
                               dtype=torch.float32)
    torch.cuda.synchronize()
    yh = G.host(y)
    for e in (0, 1, 63, 127):
        lo, hi = int(offs[e]), int(offs[e + 1])
        wo = O.quantize_weight(ws[e], "mx")
        rows = ridx[lo:hi]
        assert hi - lo > 0 and np.abs(yh[lo:hi]).max() > 0, (e, lo, hi)
        gemm_check(yh[lo:hi], O.linear(o, wo, rows=rows), O.linear_abs(o, wo, rows=rows), f"moe expert {e}")


def test_moe_bench_layout(S, G):
    """Both Qwen3-30B-A3B expert GEMMs as the benchmark launches them: each
    input prepared with the dense backbone copy alone (4:8), the grouped GEMM
    reading it.  gate/up: 4096 tokens x 2048 with RMSNorm, rows gathered by the
    router; down: the 32768 expert-sorted rows x 768, no norm, identity row
    map.  Prepared bytes against the oracle (all rows for gate/up; the rows of
    the checked experts for down -- the preparation is row-wise), the bf16
    output equal to the fp32 one rounded, every routed output written (the
    fp32 output is filled with NaN first; gate/up's 1902 (column tile, row
    tile) units are not a multiple of the 8 XCDs, so the tile order skips
    ids), and the slices of four experts (all their rows, all columns)
    against the oracle."""
    cfg = synth.MOE
    T, H, E, I, k = cfg["tokens"], cfg["hidden"], cfg["experts"], cfg["inter"], cfg["topk"]
    ridx, offs = synth.router_topk(T, E, k, seed=0)
    total = int(offs[-1])
    ri, of = torch.from_numpy(ridx).cuda(), torch.from_numpy(offs).cuda()
    experts = (0, 1, 63, 127)

    def quantized_experts(N, K, seed0):
        return S.stack_weights([S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=seed0 + e)))
                                for e in range(E)])

    # gate/up input: RMSNorm, dense backbone copy alone
    say(f"[moe-bench] gate_up T={T} K={H} N={2 * I}")
    x, g = synth.activations(T, H, seed=0), synth.gamma(H, seed=0)
    a1 = S.sharq_prepare(G.dev_bf16(x), G.dev_bf16(g), 1e-6, 4, 8, "mx",
                         out=S.alloc_act(T, H, 4, 8, "mx", "cuda", dense_only=True))
    w1 = quantized_experts(2 * I, H, 100)
    y1 = torch.full((total, 2 * I), float("nan"), dtype=torch.float32, device="cuda")
    S.sharq_linear_grouped(a1, ri, of, total, w1, out=y1)
    y1b = S.sharq_linear_grouped(a1, ri, of, total, w1, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y1).all()), "gate_up: routed outputs left unwritten"
    assert a1.sp_codes is None and a1.sp_meta is None
    o1 = O.prepare(x, g, 1e-6, 4, 8, "mx")
    dev1 = L.act_to_device_layout(o1)
    G.assert_bytes_equal("moe gate_up sp_dense", G.host(a1.sp_dense), L.dense_backbone_to_device_layout(o1))
    for name in ("sp_scale", "dn_codes", "dn_scale"):
        G.assert_bytes_equal(f"moe gate_up {name}", G.host(getattr(a1, name)), dev1[name])
    assert torch.equal(y1b, y1.to(torch.bfloat16))
    yh = G.host(y1)
    for e in experts:
        lo, hi = int(offs[e]), int(offs[e + 1])
        wo = O.quantize_weight(synth.weight(2 * I, H, seed=100 + e), "mx")
        rows = ridx[lo:hi]
        gemm_check(yh[lo:hi], O.linear(o1, wo, rows=rows), O.linear_abs(o1, wo, rows=rows), f"moe gate_up e{e}")
    del w1, y1, y1b

    # down input: expert-sorted rows, no norm, identity row map
    say(f"[moe-bench] down T={total} K={I} N={H}")
    h = synth.activations(total, I, seed=1)
    a2 = S.sharq_prepare(G.dev_bf16(h), None, 1e-6, 4, 8, "mx",
                         out=S.alloc_act(total, I, 4, 8, "mx", "cuda", dense_only=True))
    w2 = quantized_experts(H, I, 1000)
    y2 = torch.full((total, H), float("nan"), dtype=torch.float32, device="cuda")
    S.sharq_linear_grouped(a2, None, of, total, w2, out=y2)
    y2b = S.sharq_linear_grouped(a2, None, of, total, w2, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y2).all()), "down: routed outputs left unwritten"
    assert torch.equal(y2b, y2.to(torch.bfloat16))
    chk = np.concatenate([np.arange(offs[e], offs[e + 1]) for e in experts])
    o2 = O.prepare(h[chk], None, 1e-6, 4, 8, "mx")
    G.assert_bytes_equal("moe down sp_dense", L.from_panels(G.host(a2.sp_dense), total, I, I // 2)[chk],
                         L.dense_backbone_rowmajor(o2))
    for name, width in (("sp_scale", I // 32), ("dn_codes", I // 2), ("dn_scale", I // 32)):
        G.assert_bytes_equal(f"moe down {name}", L.from_panels(G.host(getattr(a2, name)), total, I, width)[chk],
                             o2[name])
    yh = G.host(y2)
    start = 0
    for e in experts:
        lo, hi = int(offs[e]), int(offs[e + 1])
        wo = O.quantize_weight(synth.weight(H, I, seed=1000 + e), "mx")
        rows = np.arange(start, start + hi - lo)
        start += hi - lo
        gemm_check(yh[lo:hi], O.linear(o2, wo, rows=rows), O.linear_abs(o2, wo, rows=rows), f"moe down e{e}")


# --------------------------------------------------------------------------- persistent kernel tail

@pytest.mark.parametrize("T,N,K,n,m", [(12750, 704, 256, 2, 4),    # 300 tiles: 44 in the last round
                                       (4608, 2048, 128, 2, 4),    # 288 tiles: 32, XCD-ordered halves
                                       (4608, 2048, 256, 4, 8)])
def test_persistent_tail_half_tiles(S, G, T, N, K, n, m):
    """A last round of at most half the CUs runs as half tiles of 128 columns
    (ragged rows and columns included): every output against the oracle, the
    bf16 output (LDS-staged epilogue) equal to the fp32 one rounded, and the
    dense backbone copy bit-identical to the compressed backbone."""
    say(f"[tail] T={T} N={N} K={K} {n}:{m}")
    x, g = synth.activations(T, K, seed=T + N), synth.gamma(K, seed=5)
    xd, gd = G.dev_bf16(x), G.dev_bf16(g)
    c = S.sharq_prepare(xd, gd, 1e-6, n, m, "mx")
    a = S.sharq_prepare(xd, gd, 1e-6, n, m, "mx", out=S.alloc_act(T, K, n, m, "mx", "cuda", dense_backbone=True))
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=K)))
    y32 = S.sharq_linear(c, wq, dtype=torch.float32)
    y16 = S.sharq_linear(c, wq, dtype=torch.bfloat16)
    yd = S.sharq_linear(a, wq, dtype=torch.float32)
    yd16 = S.sharq_linear(a, wq, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(y16, y32.to(torch.bfloat16))
    assert torch.equal(yd, y32) and torch.equal(yd16, y16)
    o = O.prepare(x, g, 1e-6, n, m, "mx")
    wo = G.weight_to_oracle(wq)
    gemm_check(G.host(y32), O.linear(o, wo), O.linear_abs(o, wo), f"tail T{T}N{N}K{K}")


@pytest.mark.parametrize("T,N,K", [(2176, 4000, 512),    # 272 tiles: 16 as half tiles; ragged last columns
                                   (300, 520, 256)])      # ragged rows and columns, one round
def test_persistent_bf16_row_pitch(S, G, T, N, K):
    """The persistent kernel's LDS-staged bf16 epilogue writing into rows
    longer than N (an output column slice): the range-checked stores land in
    the slice only (the columns past N keep their sentinel), equal to the
    contiguous fp32 output rounded, which matches the oracle."""
    say(f"[pitch] T={T} N={N} K={K}")
    x, g = synth.activations(T, K, seed=T + 7), synth.gamma(K, seed=7)
    a = S.sharq_prepare(G.dev_bf16(x), G.dev_bf16(g), 1e-6, 2, 4, "mx",
                        out=S.alloc_act(T, K, 2, 4, "mx", "cuda", dense_only=True))
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=N)))
    pitch = N + 96
    big = torch.full((T + 1, pitch), 3.0, dtype=torch.bfloat16, device="cuda")
    y32 = S.sharq_linear(a, wq, dtype=torch.float32)
    S.sharq_linear(a, wq, out=big[:T, :N])
    torch.cuda.synchronize()
    assert torch.equal(big[:T, :N], y32.to(torch.bfloat16))
    assert torch.all(big[:T, N:] == 3.0) and torch.all(big[T] == 3.0), "stores outside the slice"
    o = O.prepare(x, g, 1e-6, 2, 4, "mx")
    wo = G.weight_to_oracle(wq)
    rows = np.unique(np.concatenate([np.arange(0, T, max(1, T // 256)), [T - 1]]))
    gemm_check(G.host(y32)[rows], O.linear(o, wo, rows=rows), O.linear_abs(o, wo, rows=rows), f"pitch T{T}N{N}")


def test_grouped_bf16_row_pitch(S, G):
    """The grouped kernel's bf16 epilogue into rows longer than N, whole and
    half tiles (few units: every unit runs as two halves), ragged expert
    slices: the slice equals the contiguous fp32 output rounded, and nothing
    outside it is written."""
    T, E, topk, K, N = 300, 5, 3, 512, 200
    x = synth.activations(T, K, seed=11)
    o = O.prepare(x, synth.gamma(K, seed=11), 1e-6, 4, 8, "mx")
    wos = [O.quantize_weight(synth.weight(N, K, seed=300 + e), "mx") for e in range(E)]
    row_index, offs = synth.router_topk(T, E, topk, seed=11)
    total = int(offs[-1])
    a = G.oracle_to_act(o, dense_backbone=True)
    w = S.stack_weights([G.oracle_to_weight(wo) for wo in wos])
    ri, of = torch.from_numpy(row_index).cuda(), torch.from_numpy(offs).cuda()
    y32 = S.sharq_linear_grouped(a, ri, of, total, w, dtype=torch.float32)
    big = torch.full((total + 1, N + 40), 3.0, dtype=torch.bfloat16, device="cuda")
    S.sharq_linear_grouped(a, ri, of, total, w, out=big[:total, :N])
    torch.cuda.synchronize()
    assert torch.equal(big[:total, :N], y32.to(torch.bfloat16))
    assert torch.all(big[:total, N:] == 3.0) and torch.all(big[total] == 3.0), "stores outside the slice"
    ref = O.linear_grouped(o, row_index, offs, wos)
    yabs = np.zeros_like(ref)
    for e in range(E):
        lo, hi = offs[e], offs[e + 1]
        if hi > lo:
            yabs[lo:hi] = O.linear_abs(o, wos[e], rows=row_index[lo:hi])
    gemm_check(G.host(y32), ref, yabs, "grouped pitch")


# --------------------------------------------------------------------------- dense backbone copy

@pytest.mark.parametrize("T,K,N,use_gamma,n,m,pairs", [(300, 1024, 512, True, 2, 4, False),
                                                       (300, 640, 300, True, 4, 8, False),
                                                       (288, 2048, 256, False, 4, 8, True),
                                                       (40, 1024, 12544, True, 2, 4, False),
                                                       (200, 512, 12800, False, 2, 4, False),
                                                       (130, 416, 96, False, 2, 4, False)])
def test_dense_backbone_copy(S, G, T, K, N, use_gamma, n, m, pairs):
    """The optional dense backbone copy: byte-exact against the oracle's
    backbone codes, and the main GEMM on it gives bit-identically the result
    of expanding the compressed backbone (the MFMA operands are the same).
    Every case but the last reaches the persistent kernel that reads the copy
    (K a multiple of 128, and M > 256 or at least 48 tiles of 128 x 256: the
    small-M kernel takes the rest); the last (K = 416) runs the ragged-K
    kernel, which ignores the copy."""
    say(f"[dense-backbone] T={T} K={K} N={N} {n}:{m}{'p' if pairs else ''}")
    x = synth.activations(T, K, seed=K + T)
    g = synth.gamma(K, seed=3) if use_gamma else None
    xd, gd = G.dev_bf16(x), (None if g is None else G.dev_bf16(g))
    a = S.sharq_prepare(xd, gd, 1e-6, n, m, "mx", pairs=pairs, out=S.alloc_act(T, K, n, m, "mx", "cuda", pairs,
                                                                                dense_backbone=True))
    c = S.sharq_prepare(xd, gd, 1e-6, n, m, "mx", pairs=pairs)
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=N)))
    yd = S.sharq_linear(a, wq, dtype=torch.float32)
    yc = S.sharq_linear(c, wq, dtype=torch.float32)
    yd16 = S.sharq_linear(a, wq, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    o = O.prepare(x, g, 1e-6, n, m, "mx", pairs=pairs)
    G.assert_bytes_equal("sp_dense", G.host(a.sp_dense), L.dense_backbone_to_device_layout(o))
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(name, G.host(getattr(a, name)), G.host(getattr(c, name)))
    assert torch.equal(yd, yc)
    assert torch.equal(yd16, yd.to(torch.bfloat16))
    wo = G.weight_to_oracle(wq)
    gemm_check(G.host(yd), O.linear(o, wo), O.linear_abs(o, wo), f"dense-backbone T{T}")


@pytest.mark.parametrize("T,E,topk,K,N", [(300, 5, 3, 512, 200), (700, 16, 4, 768, 256)])
def test_grouped_dense_backbone(S, G, T, E, topk, K, N):
    """The grouped GEMM on the dense backbone copy: bit-identical to expanding
    the compressed backbone, and within the gate of the oracle."""
    say(f"[grouped-dense] T={T} E={E} top{topk} K={K} N={N}")
    x = synth.activations(T, K, seed=E + 1)
    xd, gd = G.dev_bf16(x), G.dev_bf16(synth.gamma(K, seed=E))
    a = S.sharq_prepare(xd, gd, 1e-6, 4, 8, "mx", out=S.alloc_act(T, K, 4, 8, "mx", "cuda", dense_backbone=True))
    c = S.sharq_prepare(xd, gd, 1e-6, 4, 8, "mx")
    w = S.stack_weights([S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=200 + e))) for e in range(E)])
    row_index, offs = synth.router_topk(T, E, topk, seed=E)
    total = int(offs[-1])
    ri, of = torch.from_numpy(row_index).cuda(), torch.from_numpy(offs).cuda()
    yd = S.sharq_linear_grouped(a, ri, of, total, w, dtype=torch.float32)
    yc = S.sharq_linear_grouped(c, ri, of, total, w, dtype=torch.float32)
    torch.cuda.synchronize()
    assert torch.equal(yd, yc)
    o = G.act_to_oracle(c)
    wos = [G.weight_to_oracle(w, e) for e in range(E)]
    ref = O.linear_grouped(o, row_index, offs, wos)
    yabs = np.zeros_like(ref)
    for e in range(E):
        lo, hi = offs[e], offs[e + 1]
        if hi > lo:
            yabs[lo:hi] = O.linear_abs(o, wos[e], rows=row_index[lo:hi])
    gemm_check(G.host(yd), ref, yabs, f"grouped-dense T{T}E{E}")
