"""Pins of the oracle's path combinations (Sec. 4.4, table
"ablation-combination"; Sec. 3.1 eq. "direct-sparse-quant"; the RTN rows of
table "ablation-format").

Each mode is rebuilt here from independent pieces -- an exhaustive-search
FP4 quantizer per block, an exhaustive-search E4M3 rounding, a brute-force
N:M subset choice -- and compared with the oracle's prepare_mode, buffer by
buffer and value by value.  None of these tests needs a GPU.
"""

import itertools
import math
from fractions import Fraction

import numpy as np
import pytest

from oracle import sharq_oracle as O
import panel_layout as L
from paper_2606_26587_amd import synth

GRID = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
MODES = ["sharq", "sparse", "dense", "dense_dense", "sparse_sparse"]


def nearest_grid(a: float) -> float:
    """|a| -> nearest E2M1 magnitude (ties to the even code), saturating at 6."""
    fa = Fraction(a)
    c = min(range(8), key=lambda i: (abs(fa - Fraction(GRID[i])), i % 2, i))
    return GRID[c]


def plain_mx_block(blk):
    """One MXFP4 block by exhaustive search: scale 2^(floor(log2 amax) - 2)."""
    blk = [float(v) for v in blk]
    amax = max(abs(v) for v in blk)
    e = -127 if amax == 0 else max(math.frexp(amax)[1] - 1 - 2, -127)
    s = math.ldexp(1.0, e)
    return [math.copysign(nearest_grid(float(np.float32(abs(v) / s))) * s, v) for v in blk]


def e4m3_nearest(a: float) -> float:
    vals = O.e4m3_values()
    if a >= 448.0:
        return 448.0
    d = np.abs(vals - a)
    ties = np.flatnonzero(d == d.min())
    return float(vals[ties[0] if len(ties) == 1 else [t for t in ties if t % 2 == 0][0]])


def plain_nv_block(blk, S):
    """One NVFP4 block: d = E4M3(amax / (6 S)), codes of v / (d S), value (q d) S."""
    S = np.float32(S)
    amax = np.float32(max(abs(float(v)) for v in blk))
    d = np.float32(e4m3_nearest(float(np.float32(amax / np.float32(np.float32(6.0) * S)))))
    step = np.float32(d * S)
    out = []
    for v in blk:
        v = np.float32(v)
        if d == 0:
            out.append(0.0)
            continue
        q = math.copysign(nearest_grid(abs(float(np.float32(v / step)))), float(v))
        out.append(float(np.float32(np.float32(q * d) * S)))
    return out


def plain_quant(v, fmt, S=None, block=None):
    """Row-wise blocked FP4 quantization by exhaustive search (fp64 values)."""
    v = np.asarray(v, dtype=np.float32)
    block = block or (32 if fmt == "mx" else 16)
    out = np.zeros(v.shape)
    for t in range(v.shape[0]):
        for b in range(0, v.shape[1], block):
            blk = v[t, b:b + block]
            out[t, b:b + block] = plain_mx_block(blk) if fmt == "mx" else plain_nv_block(blk, S)
    return out


def brute_keep(v, n, m, pairs=False):
    """The n-subset of every group of m with the largest sum of |v| (ties:
    the lexicographically smallest index set); in pairs: n/2 whole pairs
    scored by their larger magnitude."""
    v = np.abs(np.asarray(v, dtype=np.float64))
    T, K = v.shape
    keep = np.zeros((T, K), bool)
    for t in range(T):
        for g in range(0, K, m):
            a = v[t, g:g + m]
            if pairs:
                score = [max(a[2 * i], a[2 * i + 1]) for i in range(m // 2)]
                # the best set maximizes the sorted score vector (lexicographic)
                best = max(itertools.combinations(range(m // 2), n // 2),
                           key=lambda s: (sorted((score[i] for i in s), reverse=True), [-i for i in s]))
                for i in best:
                    keep[t, g + 2 * i] = keep[t, g + 2 * i + 1] = True
            else:
                best = max(itertools.combinations(range(m), n),
                           key=lambda s: (sorted((a[i] for i in s), reverse=True), [-i for i in s]))
                for i in best:
                    keep[t, g + i] = True
    return keep


def case(fmt, T=6, K=128, seed=0, gamma=True):
    x = synth.activations(T, K, seed=seed, fixed_outliers=(3, 77), outlier_scale=50.0, massive=False)
    g = synth.gamma(K, seed) if gamma else None
    return x, g


def reference_mode(x, g, eps, n, m, fmt, mode, pairs=False):
    """A mode rebuilt from the independent pieces above: (y, d1, R, d2, keep1, keep2)."""
    y, _ = O.rmsnorm(O.bf16_bits_to_f32(x), None if g is None else O.bf16_bits_to_f32(g), eps)
    S = None if fmt == "mx" else O.pts_scale(np.abs(y).max())
    k1, k2 = O.MODE_PATHS[mode]

    def path(v, kind):
        if kind is None:
            return np.zeros(v.shape), np.zeros(v.shape, bool)
        if kind == "sparse":
            keep = brute_keep(v, n, m, pairs)
            return plain_quant(np.where(keep, v, np.float32(0)), fmt, S, 32), keep
        return plain_quant(v, fmt, S), np.ones(v.shape, bool)

    d1, keep1 = path(y, k1)
    R = (y - d1.astype(np.float32)).astype(np.float32)
    d2, keep2 = path(R, k2)
    return y, d1, R, d2, keep1, keep2


@pytest.mark.parametrize("fmt", ["mx", "nv"])
@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("n,m,pairs", [(2, 4, False), (4, 8, False), (4, 8, True)])
def test_mode_matches_independent_rebuild(fmt, mode, n, m, pairs):
    x, g = case(fmt, seed=n + m + pairs)
    o = O.prepare_mode(x, g, 1e-6, n, m, fmt, mode, pairs=pairs)
    y, d1, R, d2, keep1, keep2 = reference_mode(x, g, 1e-6, n, m, fmt, mode, pairs)
    assert np.array_equal(o["y"], y)
    assert np.array_equal(o["d_sp"].astype(np.float64), d1)
    assert np.array_equal(o["R"], R)
    assert np.array_equal(o["d_dn"].astype(np.float64), d2)
    k1, k2 = O.MODE_PATHS[mode]
    if k1 == "sparse":
        assert np.array_equal(o["keep"], keep1)
    if k2 == "sparse":
        assert np.array_equal(o["keep2"], keep2)
    # the packed buffers decode to the same values.  The GEMM operands are
    # exact products (NVFP4: q d S in fp64, where the residual used
    # fl32(fl32(q d) S)), so NVFP4 agrees to one fp32 rounding.
    a1, a2 = O.dequant_act(o)
    if fmt == "mx":
        assert np.array_equal(a1, d1) and np.array_equal(a2, d2)
    else:
        assert np.allclose(a1, d1, rtol=2.0 ** -23, atol=0) and np.allclose(a2, d2, rtol=2.0 ** -23, atol=0)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
@pytest.mark.parametrize("n,m,pairs", [(2, 4, False), (4, 8, True)])
def test_sharq_mode_is_prepare(fmt, n, m, pairs):
    x, g = case(fmt, T=5, K=256, seed=3)
    a = O.prepare(x, g, 1e-5, n, m, fmt, pairs=pairs)
    b = O.prepare_mode(x, g, 1e-5, n, m, fmt, "sharq", pairs=pairs)
    for k in O.ACT_BUFFERS:
        assert np.array_equal(a[k], b[k]), k
    assert b["dn_meta"].shape == (5, 0)


@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_dense_mode_is_the_n0_case(fmt):
    """Plain FP4 RTN equals SharQ with an empty backbone (the residual is y)."""
    x, g = case(fmt, seed=5)
    a = O.prepare(x, g, 1e-6, 0, 4, fmt)
    b = O.prepare_mode(x, g, 1e-6, 2, 4, fmt, "dense")
    assert np.array_equal(a["dn_codes"], b["dn_codes"]) and np.array_equal(a["dn_scale"], b["dn_scale"])
    assert b["sp_codes"].shape[1] == 0 and b["sp_scale"].shape[1] == 0


def test_buffer_widths_per_mode():
    K, n, m = 256, 2, 4
    for fmt in ("mx", "nv"):
        for mode in MODES:
            o = O.prepare_mode(*case(fmt, T=3, K=K, seed=1), 1e-6, n, m, fmt, mode)
            w = O.act_widths(K, n, m, fmt, mode)
            for k in O.ACT_BUFFERS_ALL:
                assert o[k].shape == (3, w[k]), (fmt, mode, k)
    assert O.act_widths(K, n, m, "nv", "dense_dense")["sp_scale"] == K // 16
    assert O.act_widths(K, n, m, "nv", "sparse_sparse")["dn_scale"] == K // 32
    assert O.act_widths(K, n, m, "mx", "sparse_sparse")["dn_meta"] == K // 8


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("K", [128, 416])
def test_mode_device_layout_roundtrip(mode, K):
    x, g = case("nv", T=9, K=K, seed=K)
    o = O.prepare_mode(x, g, 1e-6, 4, 8, "nv", mode)
    dev = L.act_to_device_layout(o)
    back = L.act_from_device_layout(dev, 9, K, 4, 8, "nv", o["tensor_scale"], mode=mode)
    for k in O.ACT_BUFFERS_ALL:
        assert np.array_equal(back[k], o[k]), k


def test_representable_input_leaves_nothing_for_the_second_path():
    """Values on the MXFP4 grid (block peak 4 or 6 times 2^e): a dense first
    path is exact and the second path quantizes zeros (E8M0 code 0)."""
    rng = np.random.default_rng(4)
    T, K = 4, 128
    mags = rng.choice(GRID, size=(T, K)) * rng.choice([-1.0, 1.0], size=(T, K))
    mags[:, ::32] = 6.0
    e = rng.integers(-4, 4, size=(T, K // 32))
    v = (mags * np.ldexp(1.0, np.repeat(e, 32, axis=1))).astype(np.float32)
    x = synth.f32_to_bf16_bits(v)
    assert np.array_equal(synth.bf16_bits_to_f32(x), v)
    o = O.prepare_mode(x, None, 1e-6, 2, 4, "mx", "dense_dense")
    assert np.array_equal(o["d_sp"], v)
    assert not np.any(o["R"]) and not np.any(o["d_dn"])
    assert np.all(o["dn_scale"] == 0)
    # a 2:4-sparse representable row: the sparse first path is exact as well
    v2 = v.copy()
    v2[:, 1::2] = 0.0
    o2 = O.prepare_mode(synth.f32_to_bf16_bits(v2), None, 1e-6, 2, 4, "mx", "sparse_sparse")
    assert np.array_equal(o2["d_sp"], v2) and not np.any(o2["d_dn"])


def test_two_path_error_identity_and_bounds():
    """Sec. 3.5's identity y - (D1 + D2) = R - D2 holds for every two-path
    mode, and a dense second path leaves at most 2^(e+1) per element."""
    x, g = case("mx", T=8, K=256, seed=2)
    for mode in ("dense_dense", "sharq"):
        o = O.prepare_mode(x, g, 1e-6, 2, 4, "mx", mode)
        y = o["y"].astype(np.float64)
        lhs = y - (o["d_sp"].astype(np.float64) + o["d_dn"].astype(np.float64))
        assert np.array_equal(lhs, o["R"].astype(np.float64) - o["d_dn"])
        e = np.repeat(O.e8m0_exponent(np.abs(o["R"]).reshape(8, -1, 32).max(axis=2)), 32, axis=1)
        assert np.all(np.abs(lhs) <= np.ldexp(2.0, e))


@pytest.mark.parametrize("mode", MODES)
@pytest.mark.parametrize("fmt", ["mx", "nv"])
def test_mode_gemm_matches_exact_sum(mode, fmt):
    """Y = sum over the mode's paths of D_p W_view^T, checked with exact
    rational sums on a subset of outputs (the operands are pinned above)."""
    c = synth.tiny_case()
    o = O.prepare_mode(c["x"], c["gamma"], c["eps"], 2, 4, fmt, mode)
    wq = O.quantize_weight(c["w"], fmt)
    Y = O.linear(o, wq)
    d1, d2 = O.dequant_act(o)
    W = O.dequant_weight(wq, "dn")
    for t in range(0, 8, 3):
        for nn in range(0, 64, 9):
            exact = sum((Fraction(float(d1[t, k])) + Fraction(float(d2[t, k]))) * Fraction(float(W[nn, k]))
                        for k in range(128))
            assert abs(float(exact) - Y[t, nn]) <= 1e-12 * max(1.0, abs(float(exact)))


def test_reconstruction_ordering_on_outliers():
    """The paper's ablation ordering, reproduced on the synthetic outlier
    activations as activation reconstruction error: dropping the residual is
    worse than plain RTN; any second path beats RTN; SharQ and Dense+Dense
    are the two best (statistical, fixed seed).  Measured (MXFP4 2:4):
    sparse 0.175, RTN 0.151, Sparse+Sparse 0.045, SharQ 0.029, Dense+Dense
    0.026."""
    x = synth.activations(64, 1024, seed=11)
    g = synth.gamma(1024, 11)
    err = {}
    for mode in MODES:
        o = O.prepare_mode(x, g, 1e-5, 2, 4, "mx", mode)
        y = o["y"].astype(np.float64)
        err[mode] = np.linalg.norm(y - o["d_sp"] - o["d_dn"]) / np.linalg.norm(y)
    assert err["sparse"] > err["dense"]
    for mode in ("sharq", "dense_dense", "sparse_sparse"):
        assert err[mode] < err["dense"], (mode, err)
    assert max(err["sharq"], err["dense_dense"]) < err["sparse_sparse"], err
