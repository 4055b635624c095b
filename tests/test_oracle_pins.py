"""Pins of the CPU oracle against what the paper and the mathematics fix.

Each test checks the oracle against something other than itself: the values
the paper prints, brute force over all candidates, a library routine, a closed
form, an identity or a bound.  None of them needs a GPU.
"""

import itertools
import json
import math
import os
from fractions import Fraction

import numpy as np
import pytest

from oracle import sharq_oracle as O
import panel_layout as L
from paper_2606_26587_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def facts():
    with open(os.path.join(GOLDEN, "paper_format_facts.json")) as f:
        return {k: v["value"] for k, v in json.load(f).items() if not k.startswith("_")}


def f32(v):
    return np.asarray(v, dtype=np.float32)


def ulps_around(vals, k=3):
    """Each value and its k fp32 neighbours on either side."""
    base = f32(vals).view(np.uint32).astype(np.int64)
    out = []
    for d in range(-k, k + 1):
        out.append((base + d).clip(0, 0x7F7FFFFF).astype(np.uint32).view(np.float32))
    return np.concatenate(out)


# ----------------------------------------------------------------------------- E2M1

def test_e2m1_value_set_is_the_papers():
    F = facts()
    dec = O.e2m1_decode(np.arange(16, dtype=np.uint8))
    assert sorted(set(np.abs(dec[1:8]).tolist())) == F["e2m1_nonzero_magnitudes"]
    assert dec[0] == 0 and np.abs(dec).max() == F["e2m1_max"]
    # negative half mirrors the positive half, -0 included
    assert np.all(dec[8:] == -dec[:8]) and np.signbit(dec[8])
    # local dynamic range log2(6/0.5) printed as 3.58 binades
    assert round(math.log2(6 / 0.5), 2) == F["local_dynamic_range_binades"]


def brute_e2m1(v):
    """Nearest grid value by exhaustive search; ties to the even code; sign kept."""
    out = []
    grid = [0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0]
    for x in np.asarray(v, dtype=np.float32).tolist():
        a = Fraction(abs(x))
        best = min(range(8), key=lambda c: (abs(a - Fraction(grid[c])), c % 2, c))
        out.append(best | (8 if math.copysign(1.0, x) < 0 else 0))
    return np.array(out, dtype=np.uint8)


def test_e2m1_encode_matches_exhaustive_nearest_even():
    mids = [0.0, 0.25, 0.5, 0.75, 1.0, 1.25, 1.5, 1.75, 2.0, 2.5, 3.0, 3.5, 4.0, 5.0, 6.0, 7.0, 7.999]
    vals = ulps_around(mids, k=2)
    rng = np.random.default_rng(1)
    vals = np.concatenate([vals, -vals, rng.uniform(-8, 8, 3000).astype(np.float32),
                           f32([1e-30, -1e-30, 0.0, -0.0, 1e-45, 9.0, 100.0, 3e38])])
    assert np.array_equal(O.e2m1_encode(vals), brute_e2m1(vals))


def test_e2m1_decode_encode_roundtrip_all_codes():
    c = np.arange(16, dtype=np.uint8)
    assert np.array_equal(O.e2m1_encode(O.e2m1_decode(c).astype(np.float32)), c)


# ----------------------------------------------------------------------------- E8M0

def test_e8m0_exponent_matches_frexp_and_normalizes_peak():
    rng = np.random.default_rng(2)
    a = np.concatenate([
        np.ldexp(rng.uniform(1, 2, 2000), rng.integers(-126, 127, 2000)).astype(np.float32),
        ulps_around([1.0, 2.0, 4.0, 8.0, 2.0 ** -126, 2.0 ** 127], k=2),
        f32([1e-45, 1e-40, 2.0 ** -130, 3.4e38]),
    ])
    a = a[a > 0]
    e = O.e8m0_exponent(a)
    ref = np.array([max(math.frexp(float(x))[1] - 1 - 2, -127) for x in a])
    assert np.array_equal(e, ref)
    # OCP rule: the block peak lands in [4, 8) on the E2M1 scale whenever unclamped
    r = a.astype(np.float64) / np.ldexp(1.0, e)
    un = e > -127
    assert np.all((r[un] >= 4) & (r[un] < 8))
    assert O.e8m0_exponent(f32([0.0]))[0] == -127


def _ceil_rule_brute_force(a: float) -> int:
    """Smallest e in [-127, 127] with a <= 6 * 2^e, by search in exact
    arithmetic (-127 for a = 0)."""
    fa = Fraction(a)
    for e in range(-127, 128):
        if fa <= 6 * Fraction(2) ** e:
            return e
    raise AssertionError(a)


def test_e8m0_ceil_rule_is_brute_force_smallest_unclipped_scale():
    """R13: e = ceil(log2(amax / 6)) against a search over every E8M0
    exponent, on values at and around the 1.5 * 2^E switch points, powers of
    two, subnormals, random magnitudes over the whole fp32 range, and the
    largest float."""
    rng = np.random.default_rng(13)
    E = rng.integers(-140, 127, size=200)
    edges = np.concatenate([np.ldexp(1.5, E), np.ldexp(1.0, E), np.ldexp(1.75, E)])
    rand = np.ldexp(rng.uniform(1.0, 2.0, 400), rng.integers(-149, 128, 400))
    a = np.concatenate([ulps_around(f32(edges[np.isfinite(edges)]), 2),
                        f32(rand[np.isfinite(f32(rand))]), f32([1e-45, 3e-39, 6.0, 12.0, 3.4028235e38])])
    a = a[(a > 0) & np.isfinite(a)]
    got = O.e8m0_exponent(a, "ceil")
    for v, e in zip(a, got):
        assert int(e) == _ceil_rule_brute_force(float(v)), (float(v), int(e))
    assert int(O.e8m0_exponent(f32([0.0]), "ceil")[0]) == -127
    # the floor rule is the ceil rule or one below it
    d = got - O.e8m0_exponent(a, "floor")
    assert set(np.unique(d)) <= {0, 1}


def test_e8m0_ceil_rule_never_clips_and_normalizes_the_peak():
    """Under the ceil rule no value of a block exceeds 6 * 2^e, so no code
    saturates, and a block peak of normal magnitude lands in (3, 6] * 2^e;
    the residual against the quantized backbone stays exact."""
    x = synth.activations(16, 1024, seed=13)
    y = O.bf16_bits_to_f32(x)
    codes, e, _, deq = O.mx_quantize(y, None, "ceil")
    peak = np.abs(y).reshape(16, 32, 32).max(axis=2)
    scaled = peak / np.ldexp(1.0, e)
    assert np.all(scaled <= 6.0) and np.all(scaled > 3.0)
    # a value rounds to the nearest E2M1 magnitude without saturating: the
    # error is at most half the grid step at its magnitude (1 between 4 and 6)
    err = np.abs(deq.astype(np.float64) - y) / np.ldexp(1.0, np.repeat(e, 32, axis=1))
    assert err.max() <= 1.0
    o = O.prepare(x, None, 1e-6, 2, 4, "mx", scale_rule="ceil")
    assert np.array_equal((o["d_sp"] + o["R"]).astype(np.float32), y)


def test_pow2_f32_exact():
    for e in list(range(-149, 128)):
        assert float(O.pow2_f32(np.array([e]))[0]) == math.ldexp(1.0, e)


# ----------------------------------------------------------------------------- mask

def exact_sum(vals):
    return sum(Fraction(float(v)) for v in vals)


@pytest.mark.parametrize("n,m", [(2, 4), (4, 8), (1, 4), (3, 8)])
def test_mask_is_brute_force_best_subset(n, m):
    rng = np.random.default_rng(3 + n + m)
    # small-integer magnitudes force many ties; random floats exercise the general case
    y = np.concatenate([rng.integers(-3, 4, size=(200, m)).astype(np.float32),
                        rng.standard_normal((200, m)).astype(np.float32)], axis=0)
    keep = O.nm_mask(y, n, m)
    for row, k in zip(y, keep):
        best = max(itertools.combinations(range(m), n),
                   key=lambda S: (exact_sum(np.abs(row[list(S)])), [-i for i in S]))
        assert tuple(np.nonzero(k)[0]) == best


def test_mask_exactly_n_and_keeps_group_max():
    x = synth.activations(16, 256, seed=5)
    y = O.bf16_bits_to_f32(x)
    for n, m in [(2, 4), (4, 8)]:
        keep = O.nm_mask(y, n, m)
        g = keep.reshape(16, -1, m)
        assert np.all(g.sum(axis=2) == n)
        a = np.abs(y).reshape(16, -1, m)
        first_max = np.argmax(a, axis=2)   # lowest index among equal maxima
        assert np.all(np.take_along_axis(g, first_max[..., None], axis=2))


def test_pair_mask_is_brute_force_dominant_pair_set():
    """4:8 in pairs (App. A.1.4): of the 6 ways to keep 2 of the 4 pairs, the
    kept one is the only set whose every pair outranks every dropped pair
    (larger score max(|y_2i|, |y_2i+1|), or equal score and lower pair)."""
    rng = np.random.default_rng(11)
    y = np.concatenate([rng.integers(-3, 4, size=(300, 8)).astype(np.float32),
                        rng.standard_normal((300, 8)).astype(np.float32)], axis=0)
    keep = O.nm_pair_mask(y, 4, 8)
    for row, k in zip(y, keep):
        score = [max(abs(float(row[2 * i])), abs(float(row[2 * i + 1]))) for i in range(4)]
        outranks = lambda i, j: score[i] > score[j] or (score[i] == score[j] and i < j)
        dominant = [S for S in itertools.combinations(range(4), 2)
                    if all(outranks(i, j) for i in S for j in range(4) if j not in S)]
        assert len(dominant) == 1
        want = np.zeros(8, dtype=bool)
        for i in dominant[0]:
            want[2 * i] = want[2 * i + 1] = True
        assert np.array_equal(k, want)


def test_pair_mask_whole_pairs_and_group_max():
    x = synth.activations(16, 256, seed=6)
    y = O.bf16_bits_to_f32(x)
    keep = O.nm_pair_mask(y, 4, 8)
    g = keep.reshape(16, -1, 8)
    assert np.all(g.sum(axis=2) == 4)
    assert np.array_equal(g[..., 0::2], g[..., 1::2])          # whole pairs
    a = np.abs(y).reshape(16, -1, 8)
    first_max = np.argmax(a, axis=2)
    assert np.all(np.take_along_axis(g, first_max[..., None], axis=2))


def test_pair_mask_reduces_to_plain_4of8_on_equal_pairs():
    """When both elements of every pair have the same magnitude and the pair
    magnitudes are distinct, the top 2 pairs are exactly the top 4 elements."""
    rng = np.random.default_rng(12)
    mags = np.stack([rng.permutation(4) + 1.0 for _ in range(500)]).astype(np.float32)   # distinct per group
    y = np.repeat(mags, 2, axis=1) * rng.choice([-1.0, 1.0], size=(500, 8)).astype(np.float32)
    assert np.array_equal(O.nm_pair_mask(y, 4, 8), O.nm_mask(y, 4, 8))


def test_prepare_in_pairs_backbone_and_residual():
    """NVFP4 with 4:8 in pairs (the paper's primary instantiation): the packed
    backbone round-trips to whole pairs, the backbone scale equals the dense
    block scale (the group maximum is kept), and y = d_sp + R exactly where R
    is the residual before its own quantization."""
    x = synth.activations(12, 256, seed=7)
    g = synth.gamma(256, seed=7)
    for fmt in ("nv", "mx"):
        o = O.prepare(x, g, 1e-6, 4, 8, fmt, pairs=True)
        dense, keep = O.unpack_backbone(o["sp_codes"], o["sp_meta"], 256, 4, 8)
        assert np.array_equal(keep, o["keep"])
        kk = keep.reshape(12, -1, 8)
        assert np.array_equal(kk[..., 0::2], kk[..., 1::2])
        assert np.array_equal(o["R"][~keep], o["y"][~keep])
        if fmt == "mx":   # exact residual and the dense block scale (Sterbenz, group max kept)
            y = o["y"].astype(np.float64)
            assert np.array_equal(y, o["d_sp"].astype(np.float64) + o["R"].astype(np.float64))
            dense_e = O.e8m0_exponent(np.abs(o["y"]).reshape(12, -1, 32).max(axis=2))
            assert np.array_equal(o["sp_scale"].astype(np.int64) - 127, dense_e)


# ----------------------------------------------------------------------------- fused residual add

def _bf16_value(u):
    return Fraction(float(np.array([int(u) << 16], dtype=np.uint32).view(np.float32)[0]))


def _bf16_round_exact(v: Fraction) -> int:
    """Nearest bf16 to an exact rational (ties to the even pattern), by search
    over the finite bf16 values around it."""
    f = float(v)
    u = int(np.array([f], dtype=np.float32).view(np.uint32)[0]) >> 16
    cands = {c & 0xFFFF for c in (u - 1, u, u + 1, u + 2)}
    cands = [c for c in cands if (c & 0x7F80) != 0x7F80]
    best = min(cands, key=lambda c: (abs(_bf16_value(c) - v), c & 1))
    return best


def test_residual_add_is_the_correctly_rounded_bf16_sum():
    """h = bf16(fp32(x) + fp32(res)) equals the bf16 value nearest to the exact
    sum (ties to even): the fp32 intermediate never double-rounds for two
    bf16 operands."""
    rng = np.random.default_rng(31)
    n = 4000
    e1 = rng.integers(-20, 20, n)
    e2 = e1 + rng.integers(-30, 30, n)
    m1, m2 = rng.integers(128, 256, n), rng.integers(128, 256, n)
    x = (np.sign(rng.standard_normal(n)) * m1 * np.exp2(e1 - 7.0)).astype(np.float32)
    r = (np.sign(rng.standard_normal(n)) * m2 * np.exp2(e2 - 7.0)).astype(np.float32)
    xb = (x.view(np.uint32) >> 16).astype(np.uint16)
    rb = (r.view(np.uint32) >> 16).astype(np.uint16)
    # exact ties and cancellations: 1 + 2^-8, subnormals, opposite signs
    xb = np.concatenate([xb, np.array([0x3F80, 0x3F81, 0x0001, 0x4000, 0x8000], np.uint16)])
    rb = np.concatenate([rb, np.array([0x3B80, 0x3B80, 0x0001, 0xC000, 0x0000], np.uint16)])
    h = O.residual_add_bf16(xb, rb)
    for a, b, got in zip(xb, rb, h):
        want = _bf16_round_exact(_bf16_value(a) + _bf16_value(b))
        assert int(got) == want or (_bf16_value(got) == 0 and _bf16_value(want) == 0), (hex(a), hex(b), hex(got), hex(want))


def test_prepare_residual_is_prepare_of_the_sum():
    x = synth.activations(8, 256, seed=8)
    res = synth.activations(8, 256, seed=9)
    g = synth.gamma(256, seed=8)
    o = O.prepare_residual(x, res, g, 1e-6, 2, 4, "mx")
    p = O.prepare(O.residual_add_bf16(x, res), g, 1e-6, 2, 4, "mx")
    for k in O.ACT_BUFFERS:
        assert np.array_equal(o[k], p[k])


# ----------------------------------------------------------------------------- RMSNorm

def test_rms_tree_equals_recursive_traversal():
    rng = np.random.default_rng(4)
    for K in (32, 96, 128, 1000 - 8, 4096, 3584):
        x = rng.standard_normal((3, K)).astype(np.float32) * 7

        def rec(v, lo, size):
            if size == 1:
                return np.float32(v[lo] * v[lo]) if lo < len(v) else np.float32(0)
            h = size // 2
            return np.float32(rec(v, lo, h) + rec(v, lo + h, h))

        L = 1 << (K - 1).bit_length()
        ss = O.rms_sum_sq_tree(x)
        for t in range(3):
            assert ss[t].tobytes() == rec(x[t], 0, L).tobytes()


def test_rms_reciprocal_close_to_exact():
    rng = np.random.default_rng(6)
    for K in (128, 4096, 14336):
        x = (rng.standard_normal((4, K)) * rng.uniform(0.1, 30, (4, 1))).astype(np.float32)
        eps = 1e-5
        r = O.rms_reciprocal(O.rms_sum_sq_tree(x), K, eps)
        for t in range(4):
            exact = 1.0 / math.sqrt(math.fsum(float(v) * float(v) for v in x[t]) / K + float(np.float32(eps)))
            # fp32 tree error <= ceil(log2 K) half-ulps relative on ss, halved by the sqrt, plus final rounding
            bound = 0.5 * math.ceil(math.log2(K)) * 2.0 ** -24 + 2.0 ** -24
            assert abs(float(r[t]) - exact) <= bound * exact * 1.01


def test_no_gamma_is_identity():
    x = synth.activations(4, 64, seed=1)
    y, _ = O.rmsnorm(O.bf16_bits_to_f32(x), None, 1e-6)
    assert np.array_equal(y, O.bf16_bits_to_f32(x))


# ----------------------------------------------------------------------------- decomposition

def prep_tiny(n=2, m=4, fmt="mx", seed=0, T=8, K=128):
    x = synth.activations(T, K, seed=seed, fixed_outliers=(3, 77), outlier_scale=50.0, massive=False)
    return O.prepare(x, synth.gamma(K, seed), 1e-6, n, m, fmt)


@pytest.mark.parametrize("n,m", [(2, 4), (4, 8)])
def test_residual_is_exact_against_quantized_backbone(n, m):
    x = synth.activations(32, 512, seed=7)
    a = O.prepare(x, synth.gamma(512, 7), 1e-5, n, m)
    y, d_sp, R, keep = a["y"], a["d_sp"], a["R"], a["keep"]
    # eq. sharq-residual: R = X - X~_sp, and for MXFP4 the fp32 subtraction is exact
    assert np.array_equal((d_sp.astype(np.float64) + R.astype(np.float64)), y.astype(np.float64))
    assert np.array_equal(R[~keep].view(np.uint32), y[~keep].view(np.uint32))
    assert np.all(d_sp[~keep] == 0)


def test_error_identity_and_elementwise_bound():
    a = prep_tiny()
    y = a["y"].astype(np.float64)
    lhs = y - (a["d_sp"].astype(np.float64) + a["d_dn"].astype(np.float64))
    rhs = a["R"].astype(np.float64) - a["d_dn"].astype(np.float64)
    assert np.array_equal(lhs, rhs)   # Sec. 3.5 identity X - (X~_sp + R~) = R - R~
    # |R - R~| < 2 * 2^e' per element (<= 2^e' unless the element saturates at 6)
    e = np.repeat(O.e8m0_exponent(np.abs(a["R"]).reshape(a["rows"], -1, 32).max(axis=2)), 32, axis=1)
    step = np.ldexp(1.0, e)
    assert np.all(np.abs(rhs) < 2 * step)
    unsat = np.abs(a["R"]) / step <= 6
    assert np.all(np.abs(rhs)[unsat] <= step[unsat])


def test_output_perturbation_bound():
    case = synth.tiny_case()
    a = O.prepare(case["x"], case["gamma"], case["eps"], 2, 4)
    wq = O.quantize_weight(case["w"])
    Wbar = O.dequant_weight(wq)
    y = a["y"].astype(np.float64)
    lhs = np.linalg.norm(y @ Wbar.T - O.linear(a, wq))
    rhs = np.linalg.norm(a["R"].astype(np.float64) - a["d_dn"].astype(np.float64)) * np.linalg.norm(Wbar, 2)
    assert lhs <= rhs * (1 + 1e-12)


def plain_mxfp4(v):
    """Independent per-block MXFP4 round-to-nearest (OCP floor scale, nearest-even grid search)."""
    v = np.asarray(v, dtype=np.float32)
    out = np.zeros(v.shape, dtype=np.float64)
    grid = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])
    for t in range(v.shape[0]):
        for b in range(0, v.shape[1], 32):
            blk = v[t, b:b + 32].astype(np.float64)
            amax = np.abs(blk).max()
            e = -127 if amax == 0 else max(math.frexp(amax)[1] - 1 - 2, -127)
            s = math.ldexp(1.0, e)
            for j, x in enumerate(blk):
                a = abs(x) / s
                d = np.abs(grid - a)
                ties = np.flatnonzero(d == d.min())
                c = int(ties[0]) if len(ties) == 1 else int([i for i in ties if i % 2 == 0][0])
                out[t, b + j] = math.copysign(grid[c] * s, x)
    return out


def test_n0_reduces_to_plain_mxfp4():
    case = synth.tiny_case()
    a = O.prepare(case["x"], case["gamma"], case["eps"], 0, 4)
    assert np.all(a["d_sp"] == 0)
    assert np.array_equal(a["R"], a["y"])
    assert np.array_equal(a["d_dn"].astype(np.float64), plain_mxfp4(a["y"]))


def test_nm_equal_reduces_backbone_to_plain_mxfp4():
    case = synth.tiny_case()
    y = O.rmsnorm(O.bf16_bits_to_f32(case["x"]), O.bf16_bits_to_f32(case["gamma"]), case["eps"])[0]
    keep = O.nm_mask(y, 8, 8)
    assert keep.all()
    _, _, _, d_sp = O.mx_quantize(y, keep)
    assert np.array_equal(d_sp.astype(np.float64), plain_mxfp4(y))


def test_dropping_dense_path_is_direct_sparse_quant():
    """eq. direct-sparse-quant: GEMM(Q(M o X), Q(W)), computed independently."""
    case = synth.tiny_case()
    a = O.prepare(case["x"], case["gamma"], case["eps"], 2, 4)
    wq = O.quantize_weight(case["w"])
    a_sp, _ = O.dequant_act(a)
    masked = np.where(a["keep"], a["y"], np.float32(0)).astype(np.float32)
    w = O.bf16_bits_to_f32(case["w"])
    direct = plain_mxfp4(masked) @ plain_mxfp4(w).T
    assert np.allclose(a_sp @ O.dequant_weight(wq).T, direct, rtol=1e-12, atol=1e-12)


def test_sharq_beats_plain_mxfp4_on_outliers():
    """Outlier isolation (Sec. 3.5): reconstruction error below plain MXFP4's (statistical)."""
    x = synth.activations(64, 1024, seed=11)
    a = O.prepare(x, synth.gamma(1024, 11), 1e-5, 2, 4)
    y = a["y"].astype(np.float64)
    err_sharq = np.linalg.norm(y - a["d_sp"] - a["d_dn"])
    err_mx = np.linalg.norm(y - O.mx_quantize(a["y"])[3])
    assert err_sharq < 0.5 * err_mx


# ----------------------------------------------------------------------------- packing / storage

@pytest.mark.parametrize("n,m", [(2, 4), (4, 8)])
def test_backbone_pack_roundtrip(n, m):
    a = prep_tiny(n, m)
    dense, keep = O.unpack_backbone(a["sp_codes"], a["sp_meta"], a["K"], n, m)
    assert np.array_equal(keep, a["keep"])
    codes_from_deq = O.e2m1_encode(
        (a["d_sp"] / O.pow2_f32(np.repeat(a["sp_scale"].astype(np.int64) - 127, 32, axis=1))).astype(np.float32))
    assert np.array_equal(dense[keep] & 7, codes_from_deq[keep] & 7)
    assert a["sp_codes"].shape[1] == a["K"] * n // m // 2 and a["sp_meta"].shape[1] == a["K"] // 8


def test_storage_costs_match_paper():
    F = facts()
    a = prep_tiny()
    K = a["K"]
    bits = 8 * (a["dn_codes"].shape[1] + a["dn_scale"].shape[1]) / K
    assert bits == F["mxfp4_bits_per_value"] and K // a["dn_scale"].shape[1] == F["mxfp4_group"]
    nv = prep_tiny(fmt="nv")
    bits_nv = 8 * (nv["dn_codes"].shape[1] + nv["dn_scale"].shape[1]) / K
    assert bits_nv == F["nvfp4_bits_per_value"] and K // nv["dn_scale"].shape[1] == F["nvfp4_group"]


# ----------------------------------------------------------------------------- GEMM

def test_gemm_matches_exact_triple_loop():
    case = synth.tiny_case()
    a = O.prepare(case["x"], case["gamma"], case["eps"], 2, 4)
    wq = O.quantize_weight(case["w"])
    Y = O.linear(a, wq)
    a_sp, a_dn = O.dequant_act(a)
    W = O.dequant_weight(wq)
    for t in range(a["rows"]):
        for nn in range(0, wq["N"], 7):
            exact = sum(Fraction(float(a_sp[t, k])) * Fraction(float(W[nn, k])) +
                        Fraction(float(a_dn[t, k])) * Fraction(float(W[nn, k])) for k in range(a["K"]))
            assert abs(float(exact) - Y[t, nn]) <= 1e-12 * max(1.0, abs(float(exact)))


def test_grouped_equals_per_expert_linear():
    T, K, N, E = 24, 128, 48, 4
    x = synth.activations(T, K, seed=3)
    a = O.prepare(x, synth.gamma(K, 3), 1e-6, 4, 8)
    ws = [O.quantize_weight(synth.weight(N, K, seed=10 + e)) for e in range(E)]
    row_index, offs = synth.router_topk(T, E, 2, seed=3)
    Y = O.linear_grouped(a, row_index, offs, ws)
    for e in range(E):
        lo, hi = offs[e], offs[e + 1]
        ref = O.linear(a, ws[e], rows=row_index[lo:hi])
        assert np.allclose(Y[lo:hi], ref, rtol=0, atol=0)


# ----------------------------------------------------------------------------- NVFP4

def brute_e4m3(a):
    vals = O.e4m3_values()
    codes = np.arange(len(vals))   # ascending codes = ascending values
    out = []
    for x in np.asarray(a, dtype=np.float64).tolist():
        if x >= 448:
            out.append(448.0)
            continue
        d = np.abs(vals - x)
        ties = np.flatnonzero(d == d.min())
        c = ties[0] if len(ties) == 1 else [t for t in ties if codes[t] % 2 == 0][0]
        out.append(vals[c])
    return np.array(out, dtype=np.float32)


def test_e4m3_round_matches_exhaustive_nearest_even():
    vals = O.e4m3_values()
    mids = (vals[1:] + vals[:-1]) / 2
    a = np.concatenate([ulps_around(vals.astype(np.float32), 1), ulps_around(mids.astype(np.float32), 1),
                        np.random.default_rng(8).uniform(0, 500, 2000).astype(np.float32),
                        f32([0.0, 1e-10, 2.0 ** -10, 2.0 ** -9, 464.0, 465.0, 1e6])])
    a = a[a >= 0]
    assert np.array_equal(O.e4m3_round(a), brute_e4m3(a))


def test_e4m3_and_nvfp4_range_facts():
    F = facts()
    vals = O.e4m3_values()
    assert vals.max() == 448.0 and vals[vals > 0].min() == 2.0 ** -9
    lo = math.log2(0.5 * vals[vals > 0].min())
    hi = math.floor(math.log2(6 * vals.max()))
    assert [lo, hi] == F["nvfp4_binade_range"] and hi - lo + 1 == F["nvfp4_binades_total"]
    assert 6 * vals.max() == F["pts_activation_target"] == O.PTS_TARGET
    # bias 7: E4M3 value 1.0 has exponent field 7
    assert O.e4m3_encode_bits(np.array([1.0]))[0] >> 3 == F["e4m3_exponent_bias"]
    c = O.e4m3_encode_bits(vals)
    assert np.array_equal(O.e4m3_decode_bits(c), vals)


def test_nv_prepare_invariants():
    x = synth.activations(16, 256, seed=9)
    a = O.prepare(x, synth.gamma(256, 9), 1e-5, 2, 4, fmt="nv")
    S = float(a["tensor_scale"])
    assert S == float(np.float32(np.abs(a["y"]).max() / np.float32(2688)))
    d = O.e4m3_decode_bits(a["dn_scale"])
    assert np.all(np.isin(d, O.e4m3_values()))
    y = a["y"].astype(np.float64)
    assert np.array_equal(y - (a["d_sp"] + a["d_dn"].astype(np.float64)),
                          a["R"].astype(np.float64) - a["d_dn"])
    # every block peak maps close to 6 on the E2M1 scale (E4M3 normalizes within 1/16)
    Rb = np.abs(a["R"]).reshape(16, -1, 16).max(axis=2)
    ok = d > 2.0 ** -6
    ratio = Rb[ok] / (d[ok] * S)
    assert np.all((ratio > 6 * (1 - 1 / 8)) & (ratio < 6 * (1 + 1 / 8)))


def test_nv_weight_views_share_payload():
    w = synth.weight(32, 128, seed=4)
    wq = O.quantize_weight(w, "nv")
    assert np.array_equal(O.dequant_weight(wq, "sp"), O.dequant_weight(wq, "dn"))
    assert wq["scale_dn"].shape[1] == 2 * wq["scale"].shape[1]


# ----------------------------------------------------------------------------- panel layout

@pytest.mark.parametrize("K", [32, 128, 416, 4096])
def test_panel_layout_roundtrip_and_order(K):
    rng = np.random.default_rng(K)
    R = 7
    a = rng.integers(0, 256, size=(R, K // 2), dtype=np.uint8)
    flat = L.to_panels(a, K)
    assert flat.size == a.size
    assert np.array_equal(L.from_panels(flat, R, K, K // 2), a)
    # panel 0 holds row 0's first 64 bytes, then row 1's first 64 bytes, ...
    w0 = min(128, K) // 2
    assert np.array_equal(flat[:w0], a[0, :w0]) and np.array_equal(flat[w0:2 * w0], a[1, :w0])
    if K > 128:
        assert np.array_equal(flat[R * 64: R * 64 + 64 if K - 128 >= 128 else R * 64 + (K - 128) // 2],
                              a[0, 64: 128 if K - 128 >= 128 else 64 + (K - 128) // 2])


# ----------------------------------------------------------------------------- SiLU.mul fused in front (R12)

def _nearest_bf16_bits(x: float) -> int:
    """The bf16 bit pattern nearest to a finite double (ties to the even
    pattern), by search over the neighbours of its truncation."""
    sign = 0x8000 if math.copysign(1.0, x) < 0 else 0
    fx = Fraction(abs(x))
    t = (int(np.array([abs(x)], np.float32).view(np.uint32)[0]) >> 16) & 0x7FFF
    best = None
    for c in range(max(t - 2, 0), t + 3):
        v = Fraction(float(O.bf16_bits_to_f32(np.array([c], np.uint16))[0]))
        key = (abs(v - fx), c & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1] | sign


def test_exp_recipe_within_two_ulp_of_exp():
    """The recipe's e^x (R12: Cody-Waite reduction, degree-7 Taylor
    polynomial, fp32 steps) against the library exponential in fp64: within
    2 ulp of fp32 for normal results, within one subnormal step 2^-149 below
    2^-126, exact at 0, and 0 below the subnormal range."""
    rng = np.random.default_rng(21)
    x = np.concatenate([-np.abs(rng.standard_normal(50000) * 30), -rng.uniform(0, 1e-3, 2000),
                        np.linspace(-104.0, 0.0, 20001), [-0.0, -87.33654, -87.33655, -103.2789, -103.97208,
                                                          -104.5, -150.0, -1e-30]]).astype(np.float32)
    e = O.exp_nonpositive_f32(x).astype(np.float64)
    ref = np.array([math.exp(float(v)) for v in x])
    normal = ref >= 2.0 ** -126
    ulp = np.spacing(ref[normal].astype(np.float32)).astype(np.float64)
    assert np.all(np.abs(e[normal] - ref[normal]) <= 2 * ulp)
    assert np.all(np.abs(e[~normal] - ref[~normal]) <= 2.0 ** -149)
    assert float(O.exp_nonpositive_f32(np.float32(0.0))) == 1.0
    assert float(O.exp_nonpositive_f32(np.float32(-150.0))) == 0.0


def test_bf16_rounding_is_nearest_even():
    rng = np.random.default_rng(22)
    v = np.concatenate([rng.standard_normal(3000) * 10.0 ** rng.integers(-38, 38, 3000),
                        [1e-40, -3e-39, 1.00390625, 1.01171875, -2.0 ** -133]]).astype(np.float32)
    got = O.bf16_round_bits(v)
    for x, b in zip(v, got):
        assert int(b) == _nearest_bf16_bits(float(x)), (float(x), hex(int(b)))


def test_silu_mul_within_one_step_of_the_exact_product():
    """h of the fp32 recipe against bf16 of the exact SiLU(g) u: at most one
    bf16 step apart everywhere (the recipe's relative error is a few fp32 ulp,
    far below bf16's half step), and equal for almost every element; the signs
    and zeros of the special values follow the exact product."""
    rng = np.random.default_rng(12)
    g = rng.standard_normal(3000).astype(np.float32) * 4
    u = rng.standard_normal(3000).astype(np.float32) * 3
    g[:8] = [0.0, -0.0, 100.0, -100.0, -88.7, 88.7, 1e-30, -1e-30]
    u[:8] = [1.5, 2.0, -1.0, 3.0, 1.0, -2.0, 5.0, -5.0]
    gb, ub = synth.f32_to_bf16_bits(g), synth.f32_to_bf16_bits(u)
    h = O.silu_mul_bf16(gb[None], ub[None])[0]
    gf, uf = O.bf16_bits_to_f32(gb), O.bf16_bits_to_f32(ub)

    def ordinal(b):
        return -(b & 0x7FFF) if b & 0x8000 else b & 0x7FFF

    off = 0
    for i in range(3000):
        gi, ui = float(gf[i]), float(uf[i])
        sig = 1.0 / (1.0 + math.exp(-gi)) if gi > -700 else 0.0
        want = _nearest_bf16_bits(math.copysign(abs(gi * sig * ui), gi * ui) if gi * ui != 0 else
                                  (gi * 0.5) * ui)
        d = abs(ordinal(int(h[i])) - ordinal(want))
        assert d <= 1, (i, gi, ui, hex(int(h[i])), hex(want))
        off += d
    assert off <= 15, off   # a few elements within ~1e-6 of a rounding boundary
    assert [hex(int(v)) for v in h[:2]] == ["0x0", "0x8000"]


def test_prepare_silu_mul_is_prepare_of_h():
    gate, up = synth.activations(6, 256, seed=1), synth.activations(6, 256, seed=2)
    a = O.prepare_silu_mul(gate, up, 2, 4, "mx")
    b = O.prepare(a["h"], None, 0.0, 2, 4, "mx")
    for k in O.ACT_BUFFERS:
        assert np.array_equal(a[k], b[k])
