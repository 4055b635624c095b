"""NVFP4 variant of the HIP path (through the C ABI) against the CPU oracle.

Preparation, the per-tensor scales and weight quantization must match the
oracle byte for byte (the per-tensor scale as fp32 bits); the two-path GEMM
must meet the same 1e-3 accumulation gate as the MXFP4 path.
"""

import math
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


def check_prep_nv(S, G, x, g, eps, n, m, tag, ts_in=None):
    say(f"[nv-prep] {tag} shape={x.shape} n:m={n}:{m} gamma={g is not None} ts_in={ts_in}")
    xd = G.dev_bf16(x)
    gd = None if g is None else G.dev_bf16(g)
    tsd = None if ts_in is None else torch.tensor([ts_in], dtype=torch.float32, device="cuda")
    a = S.sharq_prepare(xd, gd, eps, n, m, "nv", tensor_scale_in=tsd)
    torch.cuda.synchronize()
    o = O.prepare(x, g, eps, n, m, "nv", tensor_scale=ts_in)
    assert f32_bits(G.host(a.tensor_scale)[0]) == f32_bits(o["tensor_scale"]), \
        (tag, float(G.host(a.tensor_scale)[0]), float(o["tensor_scale"]))
    dev = L.act_to_device_layout(o)
    for name in O.ACT_BUFFERS:
        G.assert_bytes_equal(f"{tag}:{name}", G.host(getattr(a, name)), dev[name])
    return a, o


NV_PREP_CASES = [
    # (T, K, gamma, n, m, eps)
    (8, 128, True, 2, 4, 1e-6),
    (37, 416, True, 2, 4, 1e-5),
    (37, 416, False, 2, 4, 1e-5),
    (37, 416, True, 4, 8, 1e-5),
    (3, 32, False, 2, 4, 1e-6),
    (64, 3584, True, 2, 4, 1e-6),
    (9, 18944, False, 2, 4, 1e-6),
    (130, 2048, True, 4, 8, 1e-6),
    (5, 16384, True, 2, 4, 1e-5),
]


@pytest.mark.parametrize("T,K,use_gamma,n,m,eps", NV_PREP_CASES)
def test_nv_prep_bit_exact(S, G, T, K, use_gamma, n, m, eps):
    x = synth.activations(T, K, seed=T + 3 * K)
    g = synth.gamma(K, seed=K + 1) if use_gamma else None
    check_prep_nv(S, G, x, g, eps, n, m, f"T{T}K{K}")


@pytest.mark.parametrize("ts", [0.02, 1.0, 3.0e-4])
def test_nv_prep_given_tensor_scale(S, G, ts):
    """A caller-supplied S (e.g. calibrated offline) is used as is and copied out."""
    x = synth.activations(20, 512, seed=11)
    check_prep_nv(S, G, x, synth.gamma(512, seed=2), 1e-6, 2, 4, f"ts{ts}", ts_in=ts)


@pytest.mark.parametrize("kind", ["zeros", "ties", "huge", "mixed", "onehot"])
@pytest.mark.parametrize("n,m", [(2, 4), (4, 8)])
def test_nv_prep_edge_values(S, G, kind, n, m):
    T, K = 12, 256
    rng = np.random.default_rng(len(kind))
    if kind == "zeros":          # all-zero tensor: S = 1, every block scale 0
        x = np.zeros((T, K), np.float32)
        x[:, ::3] = -0.0
    elif kind == "ties":
        x = rng.integers(-3, 4, size=(T, K)).astype(np.float32)
    elif kind == "huge":
        x = (rng.standard_normal((T, K)) * 1e30).astype(np.float32)
    elif kind == "mixed":        # blocks whose E4M3 scale underflows to 0 next to large ones
        x = rng.standard_normal((T, K)).astype(np.float32)
        x[0] = 0.0
        x[1, ::2] = 1e-30
        x[2] *= 1e6
        x[3, 5::7] = 6000.0
    else:                        # one large value per row: its block saturates, others are tiny
        x = (rng.standard_normal((T, K)) * 1e-3).astype(np.float32)
        x[np.arange(T), rng.integers(0, K, T)] = 5000.0
    check_prep_nv(S, G, synth.f32_to_bf16_bits(x), None, 1e-6, n, m, f"nv-edge-{kind}")


def test_nv_prep_empty(S, G):
    x = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    a = S.sharq_prepare(x, None, 1e-6, 2, 4, "nv")
    torch.cuda.synchronize()
    assert a.rows == 0


@pytest.mark.parametrize("N,K,dt", [(64, 128, "bf16"), (200, 416, "bf16"), (3584, 3584, "bf16"),
                                    (33, 18944, "bf16"), (96, 256, "f32")])
def test_nv_weight_quant_bit_exact(S, G, N, K, dt):
    say(f"[nv-wquant] N={N} K={K} {dt}")
    w = synth.weight(N, K, seed=N + 1)
    wd = G.dev_bf16(w) if dt == "bf16" else torch.from_numpy(O.bf16_bits_to_f32(w)).cuda()
    q = S.sharq_quantize_weight(wd, "nv")
    torch.cuda.synchronize()
    wo = O.quantize_weight(w, "nv")
    o = L.weight_to_device_layout(wo)
    assert f32_bits(G.host(q.tensor_scale)[0]) == f32_bits(wo["tensor_scale"])
    for name in O.WEIGHT_BUFFERS:
        G.assert_bytes_equal(name, G.host(getattr(q, name)[0]), o[name])


def gemm_check(y_gpu, y_ref, y_abs, tag):
    gate = O.gemm_gate_error(y_gpu, y_ref, y_abs)
    norm = float(np.abs(y_gpu.astype(np.float64) - y_ref).max() / max(np.abs(y_ref).max(), 1e-300))
    say(f"[nv-gemm] {tag}: gate={gate:.3e} normwise={norm:.3e}")
    assert gate <= GATE, (tag, gate)
    assert norm <= GATE, (tag, norm)


NV_LINEAR_CASES = [
    # (T, N, K, n, m)
    (8, 64, 128, 2, 4),
    (300, 200, 416, 2, 4),
    (1, 256, 3584, 2, 4),
    (129, 300, 640, 4, 8),
    (256, 512, 2048, 2, 4),
    (16, 3584, 18944, 2, 4),
]


@pytest.mark.parametrize("T,N,K,n,m", NV_LINEAR_CASES)
def test_nv_linear_parity(S, G, T, N, K, n, m):
    say(f"[nv-linear] T={T} N={N} K={K} {n}:{m}")
    x = synth.activations(T, K, seed=T + 5)
    o = O.prepare(x, synth.gamma(K, seed=3), 1e-6, n, m, "nv")
    wo = O.quantize_weight(synth.weight(N, K, seed=N + 7), "nv")
    a, w = G.oracle_to_act(o), G.oracle_to_weight(wo)
    y32 = S.sharq_linear(a, w, dtype=torch.float32)
    y16 = S.sharq_linear(a, w, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    gemm_check(G.host(y32), O.linear(o, wo), O.linear_abs(o, wo), f"T{T}N{N}K{K}")
    assert torch.equal(y16, y32.to(torch.bfloat16))


def test_nv_end_to_end_on_device(S, G):
    """Prep + quantize + GEMM all on the device, checked against the oracle run on the same inputs."""
    T, N, K = 96, 320, 1024
    x = synth.activations(T, K, seed=21)
    g = synth.gamma(K, seed=21)
    w = synth.weight(N, K, seed=21)
    a = S.sharq_prepare(G.dev_bf16(x), G.dev_bf16(g), 1e-6, 4, 8, "nv")
    wq = S.sharq_quantize_weight(G.dev_bf16(w), "nv")
    y = S.sharq_linear(a, wq, dtype=torch.float32)
    torch.cuda.synchronize()
    o = O.prepare(x, g, 1e-6, 4, 8, "nv")
    wo = O.quantize_weight(w, "nv")
    gemm_check(G.host(y), O.linear(o, wo), O.linear_abs(o, wo), "e2e")


QWEN_T = 4096


@pytest.mark.parametrize("name", ["gate_up", "down"])
def test_qwen_full_shape_nv(S, G, name):
    """Full M=4096 Qwen2.5-7B shapes: preparation compared in full, the GEMM on
    256 sampled rows x all columns, and every output written (the output is
    filled with NaN first: the persistent kernel's tile order skips ids past
    the last of its 148 x 32 or 14 x 32 tiles), then the same with the
    dense-only backbone: its copy byte-exact and the output bit-identical."""
    K, N, norm = synth.QWEN_LINEARS[name]
    say(f"[qwen-nv] {name} T={QWEN_T} K={K} N={N}")
    x = synth.activations(QWEN_T, K, seed=1)
    g = synth.gamma(K, seed=1) if norm else None
    a, o = check_prep_nv(S, G, x, g, 1e-6, 2, 4, name)
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=1)), "nv")
    y = torch.full((QWEN_T, N), float("nan"), dtype=torch.float32, device="cuda")
    S.sharq_linear(a, wq, out=y)
    # the dense-only backbone (the benchmark's form): same buffers, same output
    d = S.sharq_prepare(G.dev_bf16(x), None if g is None else G.dev_bf16(g), 1e-6, 2, 4, "nv",
                        out=S.alloc_act(QWEN_T, K, 2, 4, "nv", "cuda", dense_only=True))
    yd = torch.full((QWEN_T, N), float("nan"), dtype=torch.float32, device="cuda")
    S.sharq_linear(d, wq, out=yd)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(y).all()), f"{name}: outputs left unwritten"
    G.assert_bytes_equal("sp_dense", G.host(d.sp_dense), L.dense_backbone_to_device_layout(o))
    for buf in ("sp_scale", "dn_codes", "dn_scale", "tensor_scale"):
        G.assert_bytes_equal(buf, G.host(getattr(d, buf)).view(np.uint8), G.host(getattr(a, buf)).view(np.uint8))
    assert torch.equal(yd, y), f"{name}: the dense-only backbone changes the output"
    wo = G.weight_to_oracle(wq)
    rows = np.random.default_rng(2).choice(QWEN_T, 256, replace=False)
    rows[0], rows[1] = 0, QWEN_T - 1
    gemm_check(G.host(y)[rows], O.linear(o, wo, rows=rows), O.linear_abs(o, wo, rows=rows), name)


E2M1_MAGS = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


def e4m3_positive_value(code: int) -> float:
    """The E4M3 value of a positive code, from the format's definition
    (exponent bias 7, three mantissa bits, subnormals at exponent field 0)."""
    e, m = (code >> 3) & 15, code & 7
    return m * 2.0 ** -9 if e == 0 else 2.0 ** (e - 7) * (1 + m / 8)


def dyadic_gcd(values) -> float:
    """Largest power of two dividing every value (all are dyadic rationals)."""
    def low_bit(v):
        mant, ex = math.frexp(v)
        i = int(mant * 2.0 ** 53)
        return ex - 53 + (i & -i).bit_length() - 1
    return 2.0 ** min(low_bit(v) for v in values)


NV_EXACT_SCALES = {
    # variant: (activation scale codes, weight scale codes); the other side at 1.0
    "act_lo": (range(0x01, 0x09), [0x38]),    # subnormals 2^-9..7*2^-9, and 2^-6
    "act_hi": (range(0x70, 0x7F), [0x38]),    # 128 .. 448 (the largest finite code)
    "w_lo": ([0x38], range(0x01, 0x09)),
    "w_hi": ([0x38], range(0x70, 0x7F)),
}


def nv_exact_operands(T, N, K, n, m, variant, seed):
    """An NVFP4 prepared activation and weight built from codes and E4M3
    scales at one end of the scale range, with the code magnitudes of the
    other operand limited so that every fp32 partial sum of the two-path GEMM
    is exact whatever the order: each product q_a d_a q_w d_w is a multiple
    of Q = (1/2 gcd(d_a)) (1/2 gcd(d_w)), and at most 2K of them, each below
    max|q_a d_a| max|q_w d_w|, must stay below 2^24 Q.  The dequantized
    operands q d range over [2^-10, 2688]: exact and normal in fp16 and bf16.
    Tensor scales 2^-2 and 2^3 make the epilogue's multiply exact too."""
    rng = np.random.default_rng(seed)
    a_codes, w_codes = (list(c) for c in NV_EXACT_SCALES[variant])
    da = [e4m3_positive_value(c) for c in a_codes]
    dw = [e4m3_positive_value(c) for c in w_codes]
    q = 0.25 * dyadic_gcd(da) * dyadic_gcd(dw)
    amax, wmax = 7, 7        # largest magnitude code index of each side
    extreme_act = variant.startswith("act")
    while 2 * K * E2M1_MAGS[amax] * max(da) * E2M1_MAGS[wmax] * max(dw) >= 2.0 ** 24 * q:
        if extreme_act:
            wmax -= 1
        else:
            amax -= 1
        assert min(amax, wmax) >= 1
    keep = np.zeros((T, K // m, m), bool)
    order = rng.random((T, K // m, m)).argsort(axis=2)[..., :n]
    np.put_along_axis(keep, order, True, axis=2)
    keep = keep.reshape(T, K)

    def codes(shape, mag_max):
        return (rng.integers(0, mag_max + 1, size=shape) | (rng.integers(0, 2, size=shape) << 3)).astype(np.uint8)

    def scales(shape, pool):
        return np.asarray(pool, np.uint8)[rng.integers(0, len(pool), size=shape)]

    sp = np.where(keep, codes((T, K), amax), 0).astype(np.uint8)
    sp_codes, sp_meta = O.pack_backbone(sp, keep, n, m)
    act = {"rows": T, "K": K, "n": n, "m": m, "pairs": False, "fmt": "nv", "tensor_scale": np.float32(0.25),
           "mode": "sharq", "sp_codes": sp_codes, "sp_meta": sp_meta, "sp_scale": scales((T, K // 32), a_codes),
           "dn_codes": O.pack_nibbles(codes((T, K), amax)), "dn_scale": scales((T, K // 16), a_codes),
           "dn_meta": np.zeros((T, 0), np.uint8)}
    ws = scales((N, K // 32), w_codes)
    wq = {"N": N, "K": K, "fmt": "nv", "codes": O.pack_nibbles(codes((N, K), wmax)), "scale": ws,
          "scale_dn": np.repeat(ws, 2, axis=1), "tensor_scale": np.float32(8.0)}
    return act, wq, (amax, wmax)


NV_EXACT_CASES = ([("gate_up", 2, 4, "act_hi"), ("gate_up", 2, 4, "w_lo"), ("down", 2, 4, "act_lo"),
                   ("down", 2, 4, "w_hi")]
                  + [("ragged", n, m, v) for n, m in ((2, 4), (4, 8)) for v in sorted(NV_EXACT_SCALES)]
                  + [("mid", 4, 8, v) for v in sorted(NV_EXACT_SCALES)]
                  + [("llama_qkv", 4, 8, "act_lo"), ("llama_down", 4, 8, "w_hi")])


@pytest.mark.parametrize("name,n,m,variant", NV_EXACT_CASES)
def test_nv_exact_sums(S, G, name, n, m, variant):
    """The NVFP4 GEMMs on operands whose sums are exact in fp32, with the
    activation or weight block scales at either end of the E4M3 range: the
    output must equal the oracle's exact result bit for bit.  The Qwen2.5-7B
    shapes at M = 4096 run the persistent fp16 kernel (256 sampled rows, all
    columns; each shape takes two of the four scale ranges), and so does the
    4:8 case with ragged rows and columns, and 4:8 at two Llama-3.1-8B shapes
    at M = 2048 (the NVFP4 4:8-in-pairs benchmark's); the ragged case (K not a multiple
    of 128) the bf16 one (all outputs, every range).  Each runs on the
    compressed backbone and on its dense copy (read where K is a multiple of
    128)."""
    if name in ("ragged", "mid"):
        T, K, N = (300, 416, 520) if name == "ragged" else (300, 1024, 520)
        rows = np.arange(T)
    elif name.startswith("llama_"):
        K, N, _ = synth.LLAMA_LINEARS[name[6:]]
        T = 2048
        rows = np.random.default_rng(6).choice(T, 256, replace=False)
        rows[0], rows[1] = 0, T - 1
    else:
        K, N, _ = synth.QWEN_LINEARS[name]
        T = QWEN_T
        rows = np.random.default_rng(5).choice(T, 256, replace=False)
        rows[0], rows[1] = 0, T - 1
    o, wo, mags = nv_exact_operands(T, N, K, n, m, variant, seed=K + N + len(variant))
    say(f"[nv-exact] {name} T={T} K={K} N={N} {n}:{m} {variant} code magnitude limits {mags}")
    w = G.oracle_to_weight(wo)
    y = S.sharq_linear(G.oracle_to_act(o), w, dtype=torch.float32)
    yd = S.sharq_linear(G.oracle_to_act(o, dense_backbone=True), w, dtype=torch.float32)
    torch.cuda.synchronize()
    ref = O.linear(o, wo, rows=rows)
    for tag, out in (("compressed", y), ("dense copy", yd)):
        got = G.host(out)[rows].astype(np.float64)
        bad = np.nonzero(got != ref)
        assert bad[0].size == 0, (f"{name} {variant} {tag}: {bad[0].size} outputs differ from the exact sum; "
                                  f"first at {bad[0][0]},{bad[1][0]}: {got[bad[0][0], bad[1][0]]} vs "
                                  f"{ref[bad[0][0], bad[1][0]]}")


@pytest.mark.parametrize("T,K,N,use_gamma,n,m,pairs,form", [(300, 1024, 520, True, 2, 4, False, "both"),
                                                            (300, 640, 300, True, 4, 8, False, "only"),
                                                            (288, 2048, 256, False, 4, 8, True, "only"),
                                                            (2048, 4096, 6144, True, 4, 8, True, "only"),
                                                            (37, 3584, 300, True, 2, 4, False, "only"),
                                                            (130, 416, 96, False, 2, 4, False, "both")])
def test_nv_dense_backbone(S, G, T, K, N, use_gamma, n, m, pairs, form):
    """The NVFP4 backbone's dense copy, written beside the compressed form
    ("both") or alone ("only"): byte-exact against the oracle's backbone
    expanded to all positions, the other buffers and the per-tensor scale
    unchanged, and the GEMM on it bit-identical to the GEMM on the compressed
    backbone (same fp16 operands) and within the gate of the oracle.  K = 416
    runs the ragged-K kernel, which ignores the copy."""
    say(f"[nv-dense] T={T} K={K} N={N} {n}:{m}{'p' if pairs else ''} {form}")
    x = synth.activations(T, K, seed=K + T)
    g = synth.gamma(K, seed=3) if use_gamma else None
    xd, gd = G.dev_bf16(x), (None if g is None else G.dev_bf16(g))
    a = S.sharq_prepare(xd, gd, 1e-6, n, m, "nv", pairs=pairs,
                        out=S.alloc_act(T, K, n, m, "nv", "cuda", pairs, dense_backbone=form == "both",
                                        dense_only=form == "only"))
    c = S.sharq_prepare(xd, gd, 1e-6, n, m, "nv", pairs=pairs)
    wq = S.sharq_quantize_weight(G.dev_bf16(synth.weight(N, K, seed=N)), "nv")
    yd = S.sharq_linear(a, wq, dtype=torch.float32)
    yc = S.sharq_linear(c, wq, dtype=torch.float32)
    yd16 = S.sharq_linear(a, wq, dtype=torch.bfloat16)
    torch.cuda.synchronize()
    o = O.prepare(x, g, 1e-6, n, m, "nv", pairs=pairs)
    G.assert_bytes_equal("sp_dense", G.host(a.sp_dense), L.dense_backbone_to_device_layout(o))
    names = O.ACT_BUFFERS if form == "both" else ("sp_scale", "dn_codes", "dn_scale")
    if form == "only":
        assert a.sp_codes is None and a.sp_meta is None
    for name in names:
        G.assert_bytes_equal(name, G.host(getattr(a, name)), G.host(getattr(c, name)))
    assert f32_bits(G.host(a.tensor_scale)[0]) == f32_bits(o["tensor_scale"])
    assert torch.equal(yd, yc)
    assert torch.equal(yd16, yd.to(torch.bfloat16))
    rows = np.arange(T) if T <= 512 else np.random.default_rng(3).choice(T, 256, replace=False)
    wo = G.weight_to_oracle(wq)
    gemm_check(G.host(yd)[rows], O.linear(o, wo, rows=rows), O.linear_abs(o, wo, rows=rows), f"nv-dense T{T}")
