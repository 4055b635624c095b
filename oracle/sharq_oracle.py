"""SharQ CPU oracle -- TEST INFRASTRUCTURE ONLY.

A plain, slow, NumPy implementation of what the SharQ sparse-dense FP4 linear
layer computes, written from the paper's definitions (SharQ, arXiv 2606.26587):

  * group-wise symmetric quantization with a codebook projection
    (Sec. 3.1, eq. "group-quant"), instantiated as MXFP4 (E2M1 elements with an
    E8M0 power-of-two scale per 32 values, App. A.1.1) and NVFP4 (E2M1 with an
    E4M3 scale per 16 plus a per-tensor scale, App. A.1.2-A.1.3);
  * the online N:M activation mask that keeps the top-N magnitudes of every
    group of M (Sec. 3.1 eq. "dynamic-mask", Sec. 3.3 eq. "sharq-sparse-backbone");
  * the quantized sparse backbone (Sec. 3.3 eq. "sharq-quantized-backbone") and
    the dense residual taken against the *dequantized* backbone
    (Sec. 3.3 eq. "sharq-residual");
  * the two-path output, backbone GEMM plus residual GEMM over one shared
    quantized weight (Sec. 3.3 eq. "sharq-output", Sec. 3.4);
  * RMSNorm folded into the preparation for layers that have it (Sec. 3.4,
    "Fused sparse-residual preparation"; Fig. 2).

Only tests, the package's smoke check and the benchmark's CPU-baseline leg may
import this module.  The product path never calls it; it shares no code with
the HIP library (no common tables, helpers or generators).

Precision.  Every step that decides an integer (a mask bit, a scale exponent,
an FP4 code) is evaluated in IEEE fp32 with round-to-nearest-even and no fused
multiply-add, which is the precision the kernels decide in; the paper does not
fix one.  The RMSNorm reciprocal is evaluated in fp64 and rounded once to fp32.
The GEMMs are evaluated in fp64 over exactly dequantized operands.

Readings where the paper is silent (each also listed in the design notes):
  R1  RMSNorm: sum of squares as a balanced binary tree over K padded with
      zeros to a power of two, in fp32; r = fp32(1/sqrt(fp64(ss)/K + fp64(eps)));
      y = fp32(fp32(x*r)*gamma).  Without gamma, y = x.
  R2  The normalized row is not rounded to bf16 before masking/quantizing.
  R3  Mask score is |y|; ties go to the lower index.
  R4  MXFP4 scale: OCP floor rule, e = max(floor(log2 amax) - 2, -127),
      e = -127 for an all-zero block; E2M1 saturates at 6.
  R5  E2M1 projection ties go to the even code; the sign of zero is kept.
  R6  Backbone scale blocks are 32 logical K positions.
  R7  NVFP4: per-tensor scale S = amax/2688 over the whole call (S = 1 when
      amax = 0); block scale E4M3(amax_b / (6 S)); code E2M1(y / (d_b S));
      a zero block scale gives signed-zero codes.  Backbone blocks 32 logical
      positions, residual blocks 16.  Weights: one E4M3 scale per 32 shared by
      both paths, the dense view duplicating it per 16.
  R8  NVFP4's 4:8 in pairs (App. A.1.4 "Sparsity support"; Fig. 2 "pair-topk"):
      the 8 positions of a group form 4 pairs (2i, 2i+1) and 2 whole pairs
      survive.  A pair's score is the larger magnitude of its two elements,
      so the group maximum is always kept; of equal scores the lower pair
      wins.  Metadata: the same 8-bit keep mask per group as plain 4:8.
  R9  Residual add fused into the preparation: h = bf16(fp32(x) + fp32(res)),
      each rounding to nearest even; the preparation then works on h.
  R10 Path combinations (Sec. 4.4, table "ablation-combination"; Sec. 3.1 eq.
      "direct-sparse-quant"; the RTN rows of table "ablation-format").  Every
      mode has two path slots: path 1 quantizes y, path 2 quantizes the
      residual of y against path 1's dequantized values.  A sparse path is
      the backbone quantizer (N:M mask of its own input, blocks of 32 logical
      positions); a dense path is the format's plain quantizer (MXFP4 blocks
      of 32, NVFP4 blocks of 16).  Sparse = (sparse, none); plain FP4 RTN =
      (none, dense); Dense+Dense = (dense, dense); Sparse+Sparse = (sparse,
      sparse), whose second mask is chosen on |R|; SharQ = (sparse, dense).
      NVFP4 uses one per-tensor scale S = amax(y)/2688 for both paths.
  R11 HiF4 (App. "HiFloat4 (HiF4) Data Format", Algorithm "bf16-to-hif4",
      eq. "hif4-value"): units of 64 positions along K; the algorithm runs
      on the fp32 values it is given (y, R or W) with fp32 arithmetic:
      SF = fl32(Vmax * bf16(1/7)); E6M2 = SF rounded to 2 mantissa bits
      (nearest, ties to even), clamped to [2^-48, 1.5 * 2^15] (no zero;
      the all-ones code is NaN); REC = bf16(1/1.M) * 2^-E (the 4-entry
      reciprocal table); E1_8[j] = (V8[j] * REC >= 4); E1_16[k] =
      (V16[k] * REC * 2^-E1_8[k/2] >= 2); scaled = fl32(v * REC) *
      2^-(E1_8 + E1_16); S1P2 code = nearest multiple of 1/4 (ties to even),
      saturating at 1.75, sign kept.  Element k (0-based) uses E1_8[k/8] and
      E1_16[k/4].  Value = E6M2 * 2^(E1_8 + E1_16) * S1P2.  A backbone unit
      spans 64 logical positions (dropped positions are zero).  No per-tensor
      scale.  Metadata bytes per unit: E6M2 code, E1_8 bits, E1_16 bits
      (low byte, high byte), bit j = group j.
  R12 SiLU.mul fused into the preparation of the down projection's input:
      h = bf16(SiLU(g) * u), SiLU(g) = g / (1 + exp(-g)).  The paper does not
      fix its arithmetic; it is taken as one fp32 recipe that the kernel
      evaluates identically: t = e^-|g| by Cody-Waite reduction (Cody and
      Waite, "Software Manual for the Elementary Functions", 1980) and the
      degree-7 Taylor polynomial, q = 1 + t, s = g / q (g >= 0) or
      (g t) / q (g < 0) with correctly rounded division, h = bf16(s u) to
      nearest even; every step IEEE fp32, no fused multiply-add.  The
      preparation then works on h.
  R13 E8M0 scale rule as an ablation flag (MXFP4).  Besides the OCP floor
      rule of R4, the "ceil" rule e = ceil(log2(amax / 6)): eq.
      "group-quant" sets s = amax / 6, which E8M0 cannot hold, and App. A.1.1
      notes that a power-of-two scale cannot bring every block peak to the
      E2M1 maximum; rounding s up to a power of two keeps every value within
      range (no clipping) at the price of the top binade.  It applies to both
      paths of the preparation and to the weight.

Parity unpinned.  The paper prints no worked numeric example, and for these
readings nothing it states decides between the choices, so their tests check
invariants, range facts and exhibited differences, not values the paper
fixes: the NVFP4 formula choices of R7 (pts_scale, nv_quantize: where S is
applied and the fp32 division by d S); the pair score of R8 (the larger
magnitude rather than the sum); the fp32 SF of R11 (hif4_quantize, rather
than a bf16 intermediate); the SiLU.mul recipe of R12 (silu_mul_bf16, pinned
to the exact product within one bf16 step, the recipe itself a choice).
An independent C implementation of R7 and R8 (sharq_ref.c) agrees with this
one byte for byte, which guards the code, not the reading.
"""

from __future__ import annotations

import itertools
import math

import numpy as np

# ---------------------------------------------------------------------------
# Element formats (App. A.1.2 "Format structure")
# ---------------------------------------------------------------------------

#: E2M1 magnitudes indexed by the three low code bits (App. A.1.2).
E2M1_MAGNITUDES = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0], dtype=np.float64)
E2M1_MAX = 6.0
#: NVFP4 per-tensor target, "typically 2688 for activations" (App. A.1.3).
PTS_TARGET = 2688.0
E4M3_MAX = 448.0
MX_BLOCK = 32
NV_BLOCK = 16


def bf16_bits_to_f32(u16: np.ndarray) -> np.ndarray:
    """bf16 bit patterns -> fp32 values (exact: the bf16 bits are the top half)."""
    u16 = np.asarray(u16, dtype=np.uint16)
    return (u16.astype(np.uint32) << np.uint32(16)).view(np.float32)


def e2m1_encode(v: np.ndarray) -> np.ndarray:
    """Project fp32 values onto the E2M1 grid (eq. group-quant's projection).

    Nearest representable magnitude with ties to the even code, saturating at 6;
    bit 3 of the code is the sign bit of the input (so -0 and small negatives
    give 0x8).  The thresholds below are the midpoints between neighbouring grid
    magnitudes; '>' sends a tie down (to an even code), '>=' sends it up.
    """
    v = np.asarray(v, dtype=np.float32)
    a = np.abs(v)
    mag = np.zeros(a.shape, dtype=np.uint8)
    mag += a > np.float32(0.25)   # 0 | 0.5   tie -> 0   (code 0 even)
    mag += a >= np.float32(0.75)  # 0.5 | 1   tie -> 1   (code 2 even)
    mag += a > np.float32(1.25)   # 1 | 1.5   tie -> 1   (code 2 even)
    mag += a >= np.float32(1.75)  # 1.5 | 2   tie -> 2   (code 4 even)
    mag += a > np.float32(2.5)    # 2 | 3     tie -> 2   (code 4 even)
    mag += a >= np.float32(3.5)   # 3 | 4     tie -> 4   (code 6 even)
    mag += a > np.float32(5.0)    # 4 | 6     tie -> 4   (code 6 even); > 6 saturates
    sign = np.signbit(v).astype(np.uint8) << np.uint8(3)
    return (sign | mag).astype(np.uint8)


def e2m1_decode(codes: np.ndarray) -> np.ndarray:
    """E2M1 code -> value in fp64: (-1)^(c>>3) * magnitude[c & 7]."""
    c = np.asarray(codes, dtype=np.uint8)
    mag = E2M1_MAGNITUDES[c & 7]
    return np.where((c >> 3) & 1, -mag, mag)


def _floor_log2_f32(a: np.ndarray) -> np.ndarray:
    """floor(log2 a) for positive fp32 a, read exactly from the bit pattern."""
    bits = np.asarray(a, dtype=np.float32).view(np.uint32).astype(np.int64)
    expf = (bits >> 23) & 0xFF
    mant = bits & 0x7FFFFF
    # subnormal: a = mant * 2^-149, floor(log2 a) = bit_length(mant) - 1 - 149
    # frexp(mant) = f * 2^x with f in [0.5, 1), so bit_length(mant) = x
    sub = np.frexp(np.maximum(mant, 1).astype(np.float64))[1].astype(np.int64) - 1 - 149
    return np.where(expf > 0, expf - 127, sub)


def e8m0_exponent(amax: np.ndarray, rule: str = "floor") -> np.ndarray:
    """Shared MXFP4 exponent of a block with max magnitude amax (reading R4).

    rule "floor" (the default, OCP Microscaling): e = floor(log2 amax) -
    emax(E2M1), emax = 2; the block peak may exceed 6 * 2^e and then
    saturates.  rule "ceil" (R13): e = ceil(log2(amax / 6)), the smallest
    power-of-two scale under which the peak does not exceed the E2M1 maximum
    -- eq. "group-quant"'s s = amax / 6 rounded up to a power of two, so
    nothing clips.  With E = floor(log2 amax), 6 * 2^(E-2) = 1.5 * 2^E, so
    the ceil rule is E - 2 when amax / 2^E <= 1.5 and E - 1 above.  Both are
    clamped to the E8M0 minimum -127; an all-zero block takes -127 (code 0).
    """
    amax = np.asarray(amax, dtype=np.float32)
    pos = np.where(amax > 0, amax, np.float32(1.0))
    E = _floor_log2_f32(pos)
    e = E - 2
    if rule == "ceil":
        frac = np.ldexp(pos.astype(np.float64), -E)   # amax / 2^E in [1, 2), exact
        e = e + (frac > 1.5)
    elif rule != "floor":
        raise ValueError(rule)
    e = np.maximum(e, -127)
    return np.where(amax > 0, e, -127).astype(np.int64)


def pow2_f32(e: np.ndarray) -> np.ndarray:
    """2^e as fp32 for integer e in [-149, 127] (exact, including subnormals)."""
    e = np.asarray(e, dtype=np.int64)
    out = np.where(e >= -126, ((np.clip(e, -126, 127) + 127) << 23), 1 << np.clip(e + 149, 0, 22))
    return out.astype(np.uint32).view(np.float32)


def e4m3_values() -> np.ndarray:
    """All 126 finite non-negative E4M3 values (bias 7; exponent field 0 is subnormal).

    Code (E, M): E > 0 -> 2^(E-7) (1 + M/8); E = 0 -> 2^-6 (M/8).  (E, M) = (15, 7)
    is NaN in this variant, so the largest value is 2^8 * 1.75 = 448.
    """
    vals = []
    for E in range(16):
        for M in range(8):
            if E == 15 and M == 7:
                continue
            vals.append((M / 8.0) * 2.0 ** -6 if E == 0 else (1 + M / 8.0) * 2.0 ** (E - 7))
    return np.array(vals, dtype=np.float64)


def e4m3_round(a: np.ndarray) -> np.ndarray:
    """Round non-negative fp32 values to E4M3 (nearest, ties to even mantissa, saturating at 448).

    Within binade 2^E (E >= -6) the E4M3 spacing is 2^(E-3); below 2^-6 the
    subnormal spacing is 2^-9.  Returned as fp32 (every E4M3 value is exact in fp32).
    """
    a = np.asarray(a, dtype=np.float64)
    E = np.frexp(np.where(a > 0, a, 1.0))[1].astype(np.float64) - 1   # floor(log2 a), exact
    E = np.maximum(E, -6)
    q = 2.0 ** (E - 3)
    r = np.rint(a / q) * q          # np.rint rounds half to even; a/q is exact
    r = np.minimum(r, E4M3_MAX)
    r = np.where(a > 0, r, 0.0)
    return r.astype(np.float32)


def e4m3_encode_bits(v: np.ndarray) -> np.ndarray:
    """E4M3 value (non-negative, exactly representable) -> its 8-bit code."""
    v = np.asarray(v, dtype=np.float64)
    out = np.zeros(v.shape, dtype=np.uint8)
    nz = v > 0
    E = np.frexp(np.where(nz, v, 1.0))[1].astype(np.int64) - 1
    normal = nz & (E >= -6)
    man_n = np.rint((v / 2.0 ** E - 1.0) * 8).astype(np.int64)
    out = np.where(normal, ((E + 7) << 3) | man_n, out)
    sub = nz & (E < -6)
    man_s = np.rint(v / 2.0 ** -9).astype(np.int64)
    out = np.where(sub, man_s, out)
    return out.astype(np.uint8)


def e4m3_decode_bits(c: np.ndarray) -> np.ndarray:
    c = np.asarray(c, dtype=np.int64)
    E = (c >> 3) & 15
    M = c & 7
    return np.where(E > 0, (1 + M / 8.0) * 2.0 ** (E - 7), (M / 8.0) * 2.0 ** -6)


# ---------------------------------------------------------------------------
# RMSNorm (Sec. 3.4 "Fused sparse-residual preparation", readings R1, R2)
# ---------------------------------------------------------------------------

def rms_sum_sq_tree(x: np.ndarray) -> np.ndarray:
    """Sum of squares per row as a balanced binary tree in fp32 (reading R1).

    Leaves are fl32(x_k * x_k) for k < K and zero up to the next power of two;
    every internal node is the fp32 sum of its two children.
    """
    x = np.asarray(x, dtype=np.float32)
    T, K = x.shape
    L = 1
    while L < K:
        L *= 2
    level = np.zeros((T, L), dtype=np.float32)
    level[:, :K] = x * x
    while level.shape[1] > 1:
        level = level[:, 0::2] + level[:, 1::2]
    return level[:, 0]


def rms_reciprocal(ss: np.ndarray, K: int, eps: float) -> np.ndarray:
    """r = fp32(1 / sqrt(fp64(ss)/K + fp64(eps))) with eps first rounded to fp32."""
    ss64 = np.asarray(ss, dtype=np.float32).astype(np.float64)
    eps64 = np.float64(np.float32(eps))
    return (1.0 / np.sqrt(ss64 / np.float64(K) + eps64)).astype(np.float32)


def rmsnorm(x: np.ndarray, gamma: np.ndarray | None, eps: float):
    """y = (x * r) * gamma in fp32, or y = x without gamma.  Returns (y, r)."""
    x = np.asarray(x, dtype=np.float32)
    T, K = x.shape
    if gamma is None:
        return x.copy(), np.ones(T, dtype=np.float32)
    r = rms_reciprocal(rms_sum_sq_tree(x), K, eps)
    y = (x * r[:, None]).astype(np.float32) * np.asarray(gamma, dtype=np.float32)[None, :]
    return y.astype(np.float32), r


# ---------------------------------------------------------------------------
# Online N:M mask (eq. dynamic-mask; eq. sharq-sparse-backbone; reading R3)
# ---------------------------------------------------------------------------

def nm_mask(y: np.ndarray, n: int, m: int) -> np.ndarray:
    """Keep the n largest |y| in every group of m consecutive K positions.

    rank_k = #{k' in group : |y_k'| > |y_k|, or |y_k'| == |y_k| and k' < k};
    position k is kept iff rank_k < n, so exactly n positions survive per group.
    """
    y = np.asarray(y, dtype=np.float32)
    T, K = y.shape
    a = np.abs(y).reshape(T, K // m, m)
    rank = np.zeros(a.shape, dtype=np.int64)
    for k in range(m):
        for kp in range(m):
            if kp == k:
                continue
            beats = a[..., kp] > a[..., k]
            if kp < k:
                beats = beats | (a[..., kp] == a[..., k])
            rank[..., k] += beats
    return (rank < n).reshape(T, K)


def nm_pair_mask(y: np.ndarray, n: int, m: int) -> np.ndarray:
    """n:m selection in pairs (reading R8): the m positions of a group are m/2
    adjacent pairs, and the n/2 pairs with the largest pair scores survive.

    score_i = max(|y_2i|, |y_2i+1|); pair i is kept iff
    #{j : score_j > score_i, or score_j == score_i and j < i} < n/2,
    and a kept pair keeps both of its positions.  Parity unpinned in the
    score (the larger magnitude rather than the sum).
    """
    y = np.asarray(y, dtype=np.float32)
    T, K = y.shape
    a = np.abs(y).reshape(T, K // m, m // 2, 2)
    score = a.max(axis=3)
    P = m // 2
    rank = np.zeros(score.shape, dtype=np.int64)
    for i in range(P):
        for j in range(P):
            if j == i:
                continue
            beats = score[..., j] > score[..., i]
            if j < i:
                beats = beats | (score[..., j] == score[..., i])
            rank[..., i] += beats
    keep_pair = rank < n // 2
    return np.repeat(keep_pair, 2, axis=2).reshape(T, K)


# ---------------------------------------------------------------------------
# MXFP4 block quantization (eq. group-quant with an E8M0 block scale)
# ---------------------------------------------------------------------------

def mx_quantize(vals: np.ndarray, present: np.ndarray | None = None, rule: str = "floor"):
    """Quantize rows of fp32 values to MXFP4 in blocks of 32 along K.

    `present` marks the positions that belong to the tensor (the backbone's kept
    positions); the block amax is taken over those only and the others get
    code 0.  `rule` is the E8M0 rule of e8m0_exponent.  Returns (codes uint8
    [T,K], exponent int [T,K/32], scale code uint8 [T,K/32], dequantized
    values fp32 [T,K]).
    """
    v = np.asarray(vals, dtype=np.float32)
    T, K = v.shape
    if present is None:
        present = np.ones(v.shape, dtype=bool)
    mag = np.where(present, np.abs(v), np.float32(0.0)).reshape(T, K // MX_BLOCK, MX_BLOCK)
    amax = mag.max(axis=2)
    e = e8m0_exponent(amax, rule)
    e_full = np.repeat(e, MX_BLOCK, axis=1)
    # v / 2^e: exact division by a power of two (fp32, correctly rounded);
    # positions outside `present` may overflow here and are discarded below
    with np.errstate(over="ignore"):
        scaled = (v / pow2_f32(e_full)).astype(np.float32)
    codes = np.where(present, e2m1_encode(scaled), np.uint8(0)).astype(np.uint8)
    deq = (e2m1_decode(codes) * pow2_f32(e_full).astype(np.float64)).astype(np.float32)
    deq = np.where(present, deq, np.float32(0.0)).astype(np.float32)
    return codes, e, (e + 127).astype(np.uint8), deq


# ---------------------------------------------------------------------------
# NVFP4 block quantization (App. A.1.2-A.1.3; reading R7)
# ---------------------------------------------------------------------------

def pts_scale(amax: float) -> np.float32:
    """Per-tensor scale S = fl32(amax / 2688), or 1 for an all-zero tensor.
    Parity unpinned (reading R7)."""
    amax = np.float32(amax)
    if amax == 0:
        return np.float32(1.0)
    return np.float32(amax / np.float32(PTS_TARGET))


def nv_quantize(vals: np.ndarray, S: np.float32, block: int, present: np.ndarray | None = None):
    """NVFP4 quantization of rows in blocks of `block` along K under per-tensor scale S.
    Parity unpinned (reading R7: where S is applied, the fp32 division).

    d_b = E4M3(fl32(amax_b / fl32(6 S))); code = E2M1(fl32(v / fl32(d_b S)));
    dequantized value fl32(fl32(q d_b) S).  A zero d_b gives signed-zero codes.
    Returns (codes, scale value d_b fp32 [T,K/block], scale code uint8, deq fp32).
    """
    v = np.asarray(vals, dtype=np.float32)
    T, K = v.shape
    S = np.float32(S)
    if present is None:
        present = np.ones(v.shape, dtype=bool)
    mag = np.where(present, np.abs(v), np.float32(0.0)).reshape(T, K // block, block)
    amax = mag.max(axis=2).astype(np.float32)
    six_s = np.float32(np.float32(E2M1_MAX) * S)
    d = e4m3_round((amax / six_s).astype(np.float32))
    d_full = np.repeat(d, block, axis=1)
    step = (d_full * S).astype(np.float32)
    with np.errstate(divide="ignore", invalid="ignore"):
        scaled = np.where(d_full > 0, v / np.where(step > 0, step, np.float32(1.0)), np.float32(0.0) * v)
    scaled = scaled.astype(np.float32)
    codes = e2m1_encode(scaled)
    codes = np.where(d_full > 0, codes, (np.signbit(v).astype(np.uint8) << 3)).astype(np.uint8)
    codes = np.where(present, codes, np.uint8(0)).astype(np.uint8)
    qd = (e2m1_decode(codes) * d_full.astype(np.float64)).astype(np.float32)   # exact
    deq = (qd * S).astype(np.float32)
    deq = np.where(present, deq, np.float32(0.0)).astype(np.float32)
    return codes, d, e4m3_encode_bits(d), deq


# ---------------------------------------------------------------------------
# HiF4 (App. "HiFloat4 (HiF4) Data Format"; reading R11)
# ---------------------------------------------------------------------------

HIF4_UNIT = 64
E6M2_BIAS = 48
E6M2_NAN = 0xFF
S1P2_MAX = 1.75


def bf16_round_f32(v) -> np.ndarray:
    """fp32 -> nearest bf16 value (ties to even), returned as fp32."""
    u = np.asarray(v, dtype=np.float32).view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return r.astype(np.uint32).view(np.float32)


def e6m2_decode(code) -> np.ndarray:
    """E6M2 code -> value 2^(E-48) * (1 + M/4) in fp64 (eq. "e6m2"); NaN for 0xFF."""
    c = np.asarray(code, dtype=np.int64)
    v = np.ldexp(1.0 + (c & 3) / 4.0, (c >> 2) - E6M2_BIAS)
    return np.where(c == E6M2_NAN, np.nan, v)


def e6m2_round(a) -> np.ndarray:
    """Non-negative fp32 -> E6M2 code: 2 mantissa bits, nearest with ties to
    even, clamped to the normal range [2^-48, 1.5 * 2^15] (R11)."""
    a = np.asarray(a, dtype=np.float64)
    E = np.frexp(np.where(a > 0, a, 1.0))[1].astype(np.int64) - 1          # floor(log2 a)
    q = np.rint(np.ldexp(a, -E) * 4.0)                                     # 4 * mantissa in [4, 8]
    E = np.where(q == 8, E + 1, E)
    q = np.where(q == 8, 4, q).astype(np.int64)
    code = ((E + E6M2_BIAS) << 2) | (q - 4)
    code = np.where(E > 15, (63 << 2) | 2, code)
    code = np.where((E == 15) & (q - 4 == 3), (63 << 2) | 2, code)        # 1.75 * 2^15 is the NaN code
    code = np.where((E < -E6M2_BIAS) | (a <= 0), 0, code)
    return code.astype(np.uint8)


#: bf16(1/1.M) for M = 0..3, the reciprocal table of Algorithm "bf16-to-hif4"
E6M2_REC_TABLE = bf16_round_f32(np.array([1.0, 1 / 1.25, 1 / 1.5, 1 / 1.75], dtype=np.float64).astype(np.float32))
#: bf16(1/7), the constant of the level-1 scale
ONE_SEVENTH_BF16 = bf16_round_f32(np.float32(1.0 / 7.0))


def e6m2_reciprocal(code) -> np.ndarray:
    """REC = table[M] * 2^-E in fp32 (exact scaling of the table entry)."""
    c = np.asarray(code, dtype=np.int64)
    return np.ldexp(E6M2_REC_TABLE[c & 3].astype(np.float64), -((c >> 2) - E6M2_BIAS)).astype(np.float32)


def s1p2_encode(v) -> np.ndarray:
    """Scaled fp32 -> S1P2 code: sign bit 3, magnitude m in bits 0-2 (value m/4);
    nearest multiple of 1/4 with ties to even m, saturating at 1.75."""
    v = np.asarray(v, dtype=np.float32)
    m = np.minimum(np.rint(np.abs(v).astype(np.float64) * 4.0), 7).astype(np.uint8)
    return ((np.signbit(v).astype(np.uint8) << 3) | m).astype(np.uint8)


def s1p2_decode(codes) -> np.ndarray:
    c = np.asarray(codes, dtype=np.uint8)
    mag = (c & 7).astype(np.float64) / 4.0
    return np.where((c >> 3) & 1, -mag, mag)


def hif4_quantize(vals: np.ndarray, present: np.ndarray | None = None):
    """HiF4 quantization of rows in units of 64 along K (Algorithm
    "bf16-to-hif4", reading R11; parity unpinned in its fp32 SF).  `present` marks the positions of the tensor
    (the backbone's kept ones); the others count as zero and get code 0.
    Returns (codes uint8 [T,K], meta uint8 [T,K/64*4], deq fp32 [T,K])."""
    v = np.asarray(vals, dtype=np.float32)
    T, K = v.shape
    if present is None:
        present = np.ones(v.shape, dtype=bool)
    v = np.where(present, v, np.float32(0.0)).astype(np.float32)
    U = K // HIF4_UNIT
    a = np.abs(v).reshape(T, U, HIF4_UNIT)
    v16 = a.reshape(T, U, 16, 4).max(axis=3)                 # stage 1: three-level tree of maxima
    v8 = v16.reshape(T, U, 8, 2).max(axis=3)
    vmax = v8.max(axis=2)
    sf = (vmax * ONE_SEVENTH_BF16).astype(np.float32)          # stage 2: scaling metadata
    e6 = e6m2_round(sf)
    rec = e6m2_reciprocal(e6)
    e1_8 = ((v8 * rec[..., None]).astype(np.float32) >= np.float32(4.0)).astype(np.int64)
    e8_of16 = np.repeat(e1_8, 2, axis=2)
    t16 = np.ldexp((v16 * rec[..., None]).astype(np.float32).astype(np.float64), -e8_of16)
    e1_16 = (t16 >= 2.0).astype(np.int64)
    # stage 3: scale and quantize every element
    shift = np.repeat(e1_8, 8, axis=2) + np.repeat(e1_16, 4, axis=2)
    scaled = (v.reshape(T, U, HIF4_UNIT) * rec[..., None]).astype(np.float32)
    scaled = np.ldexp(scaled.astype(np.float64), -shift).astype(np.float32)
    codes = s1p2_encode(scaled).reshape(T, K)
    codes = np.where(present, codes, np.uint8(0)).astype(np.uint8)
    meta = np.zeros((T, U, 4), dtype=np.uint8)
    meta[..., 0] = e6
    meta[..., 1] = (e1_8 << np.arange(8)).sum(axis=2).astype(np.uint8)
    b16 = (e1_16 << np.arange(16)).sum(axis=2)
    meta[..., 2] = (b16 & 0xFF).astype(np.uint8)
    meta[..., 3] = (b16 >> 8).astype(np.uint8)
    meta = meta.reshape(T, U * 4)
    return codes, meta, hif4_decode(codes, meta).astype(np.float32)


def hif4_decode(codes: np.ndarray, meta: np.ndarray) -> np.ndarray:
    """eq. "hif4-value": V_k = E6M2 * 2^(E1_8[k/8] + E1_16[k/4]) * S1P2_k (fp64, exact)."""
    c = np.asarray(codes, dtype=np.uint8)
    T, K = c.shape
    U = K // HIF4_UNIT
    m = np.asarray(meta, dtype=np.uint8).reshape(T, U, 4).astype(np.int64)
    base = e6m2_decode(m[..., 0])
    e8 = (m[..., 1:2] >> np.arange(8)) & 1
    b16 = m[..., 2] | (m[..., 3] << 8)
    e16 = (b16[..., None] >> np.arange(16)) & 1
    shift = np.repeat(e8, 8, axis=2) + np.repeat(e16, 4, axis=2)
    return (np.repeat(base, HIF4_UNIT, axis=1).reshape(T, U, HIF4_UNIT) * np.ldexp(1.0, shift)
            * s1p2_decode(c).reshape(T, U, HIF4_UNIT)).reshape(T, K)


# ---------------------------------------------------------------------------
# Packing: the compressed backbone and two codes per byte
# ---------------------------------------------------------------------------

def pack_nibbles(codes: np.ndarray) -> np.ndarray:
    """[T, 2J] 4-bit codes -> [T, J] bytes, element 2j in the low nibble."""
    c = np.asarray(codes, dtype=np.uint8)
    return (c[:, 0::2] & 0xF) | ((c[:, 1::2] & 0xF) << 4)


def unpack_nibbles(b: np.ndarray) -> np.ndarray:
    b = np.asarray(b, dtype=np.uint8)
    out = np.empty((b.shape[0], b.shape[1] * 2), dtype=np.uint8)
    out[:, 0::2] = b & 0xF
    out[:, 1::2] = b >> 4
    return out


def pack_backbone(codes: np.ndarray, keep: np.ndarray, n: int, m: int):
    """Compress the backbone: kept codes in ascending K, plus index metadata.

    m = 4, n = 2: per group the two kept positions i0 < i1 as (i0 | i1 << 2),
    two groups per byte (even group in the low nibble).
    m = 8: per group an 8-bit keep mask (bit p = position p kept).
    """
    T, K = codes.shape
    kept = codes[keep].reshape(T, K * n // m)
    sp_codes = pack_nibbles(kept)
    g = keep.reshape(T, K // m, m)
    if m == 4 and n == 2:
        pos = np.nonzero(g.reshape(-1, m))[1].reshape(T, K // m, 2)
        nib = (pos[..., 0] | (pos[..., 1] << 2)).astype(np.uint8)
        sp_meta = pack_nibbles(nib)
    elif m == 8:
        weights = (1 << np.arange(8)).astype(np.int64)
        sp_meta = (g.astype(np.int64) * weights).sum(axis=2).astype(np.uint8)
    else:
        raise ValueError(f"no metadata layout for {n}:{m}")
    return sp_codes, sp_meta


def unpack_backbone(sp_codes: np.ndarray, sp_meta: np.ndarray, K: int, n: int, m: int):
    """Inverse of pack_backbone: -> (dense codes [T,K] with 0 at pruned positions, keep)."""
    T = sp_codes.shape[0]
    kept = unpack_nibbles(sp_codes)
    keep = np.zeros((T, K // m, m), dtype=bool)
    if m == 4 and n == 2:
        nib = unpack_nibbles(sp_meta)
        i0 = nib & 3
        i1 = (nib >> 2) & 3
        t, g = np.meshgrid(np.arange(T), np.arange(K // m), indexing="ij")
        keep[t, g, i0] = True
        keep[t, g, i1] = True
    elif m == 8:
        for p in range(8):
            keep[:, :, p] = (sp_meta >> p) & 1
    else:
        raise ValueError(f"no metadata layout for {n}:{m}")
    keep = keep.reshape(T, K)
    dense = np.zeros((T, K), dtype=np.uint8)
    dense[keep] = kept.reshape(-1)
    return dense, keep


# ---------------------------------------------------------------------------
# Names and row widths of the packed buffers
# ---------------------------------------------------------------------------

ACT_BUFFERS = ("sp_codes", "sp_meta", "sp_scale", "dn_codes", "dn_scale")
#: every buffer a prepared activation may use (dn_meta: a sparse second path)
ACT_BUFFERS_ALL = ACT_BUFFERS + ("dn_meta",)
WEIGHT_BUFFERS = ("codes", "scale", "scale_dn")


def path_widths(kind, K: int, n: int, m: int, fmt: str):
    """Row bytes (codes, meta, scale) of one path slot of kind 'sparse', 'dense' or None."""
    if kind is None:
        return 0, 0, 0
    scale_sparse = K // 16 if fmt == "hif4" else K // 32
    if kind == "sparse":
        return K * n // m // 2, K // 8, scale_sparse
    return K // 2, 0, K // 32 if fmt == "mx" else K // 16


def act_widths(K: int, n: int, m: int, fmt: str, mode: str = "sharq") -> dict:
    """Row bytes of every buffer of a prepared activation in `mode` (0 = unused)."""
    k1, k2 = MODE_PATHS[mode]
    c1, m1, s1 = path_widths(k1, K, n, m, fmt)
    c2, m2, s2 = path_widths(k2, K, n, m, fmt)
    return {"sp_codes": c1, "sp_meta": m1, "sp_scale": s1, "dn_codes": c2, "dn_meta": m2, "dn_scale": s2}


# ---------------------------------------------------------------------------
# Preparation (Sec. 3.3 eqs. sharq-sparse-backbone / quantized-backbone / residual)
# ---------------------------------------------------------------------------

def prepare(x_bf16: np.ndarray, gamma_bf16: np.ndarray | None, eps: float, n: int, m: int,
            fmt: str = "mx", tensor_scale: float | None = None, pairs: bool = False,
            scale_rule: str = "floor") -> dict:
    """Activation preparation for one linear call.

    1. y = RMSNorm(x) * gamma (or y = x);
    2. keep = top-n of |y| per group of m (pairs: the top n/2 pairs, R8);
    3. backbone: quantize y on the kept positions (X_sp = M(X) o X, then Q_sp);
    4. residual R = y - D_sp(Q_sp(X_sp)), taken against the dequantized backbone;
    5. quantize R densely (Q_dn).
    scale_rule (MXFP4): the E8M0 rule of both paths, "floor" or "ceil" (R13).
    Returns the packed buffers plus debug arrays.
    """
    if scale_rule != "floor" and fmt != "mx":
        raise ValueError("the E8M0 scale rule applies to MXFP4 only")
    x = bf16_bits_to_f32(x_bf16)
    T, K = x.shape
    g = None if gamma_bf16 is None else bf16_bits_to_f32(gamma_bf16)
    y, r = rmsnorm(x, g, eps)
    if n == 0:
        keep = np.zeros(y.shape, dtype=bool)
    elif pairs:
        keep = nm_pair_mask(y, n, m)
    else:
        keep = nm_mask(y, n, m)
    out = {"rows": T, "K": K, "n": n, "m": m, "pairs": pairs, "fmt": fmt, "y": y, "r": r, "keep": keep}
    if fmt == "mx":
        sp_c, _, sp_s, d_sp = mx_quantize(y, keep, scale_rule)
        R = (y - d_sp).astype(np.float32)
        dn_c, _, dn_s, d_dn = mx_quantize(R, None, scale_rule)
        out["tensor_scale"] = None
        out["scale_rule"] = scale_rule
    elif fmt == "nv":
        if tensor_scale is None:
            S = pts_scale(np.abs(y).max() if y.size else 0.0)
        else:
            S = np.float32(tensor_scale)
        sp_c, _, sp_s, d_sp = nv_quantize(y, S, MX_BLOCK, keep)
        R = (y - d_sp).astype(np.float32)
        dn_c, _, dn_s, d_dn = nv_quantize(R, S, NV_BLOCK)
        out["tensor_scale"] = np.float32(S)
    elif fmt == "hif4":
        sp_c, sp_s, d_sp = hif4_quantize(y, keep)
        R = (y - d_sp).astype(np.float32)
        dn_c, dn_s, d_dn = hif4_quantize(R)
        out["tensor_scale"] = None
    else:
        raise ValueError(fmt)
    if n > 0:
        out["sp_codes"], out["sp_meta"] = pack_backbone(sp_c, keep, n, m)
    else:
        out["sp_codes"] = np.zeros((T, 0), np.uint8)
        out["sp_meta"] = np.zeros((T, 0), np.uint8)
    out.update(sp_scale=sp_s, dn_codes=pack_nibbles(dn_c), dn_scale=dn_s,
               d_sp=d_sp, R=R, d_dn=d_dn)
    return out


# ---------------------------------------------------------------------------
# Path combinations (Sec. 4.4 table "ablation-combination"; reading R10)
# ---------------------------------------------------------------------------

#: The kinds of the two path slots of every mode.  Path 1 quantizes y; path 2
#: quantizes the residual of y against path 1's dequantized values.
MODE_PATHS = {
    "sharq": ("sparse", "dense"),
    "sparse": ("sparse", None),
    "dense": (None, "dense"),
    "dense_dense": ("dense", "dense"),
    "sparse_sparse": ("sparse", "sparse"),
}
#: the numbering of the modes at the library's C interface
MODE_IDS = {"sharq": 0, "sparse": 1, "dense": 2, "dense_dense": 3, "sparse_sparse": 4}


def quantize_path(v: np.ndarray, kind: str, n: int, m: int, fmt: str, S, pairs: bool = False) -> dict:
    """One path applied to rows v: a sparse path keeps the top n of every m
    (of |v|, or in pairs) and quantizes the kept values in blocks of 32
    logical positions (eq. sharq-quantized-backbone); a dense path is the
    format's plain quantizer (MXFP4 blocks of 32, NVFP4 blocks of 16)."""
    T, K = v.shape
    if kind == "sparse":
        if n == 0:
            keep = np.zeros(v.shape, dtype=bool)
        else:
            keep = nm_pair_mask(v, n, m) if pairs else nm_mask(v, n, m)
        if fmt == "mx":
            c, _, sc, deq = mx_quantize(v, keep)
        elif fmt == "hif4":
            c, sc, deq = hif4_quantize(v, keep)
        else:
            c, _, sc, deq = nv_quantize(v, S, MX_BLOCK, keep)
        if n > 0:
            codes, meta = pack_backbone(c, keep, n, m)
        else:
            codes, meta = np.zeros((T, 0), np.uint8), np.zeros((T, 0), np.uint8)
        return {"codes": codes, "meta": meta, "scale": sc, "deq": deq, "keep": keep}
    if fmt == "mx":
        c, _, sc, deq = mx_quantize(v)
    elif fmt == "hif4":
        c, sc, deq = hif4_quantize(v)
    else:
        c, _, sc, deq = nv_quantize(v, S, NV_BLOCK)
    return {"codes": pack_nibbles(c), "meta": np.zeros((T, 0), np.uint8), "scale": sc, "deq": deq,
            "keep": np.ones(v.shape, dtype=bool)}


def prepare_mode(x_bf16: np.ndarray, gamma_bf16: np.ndarray | None, eps: float, n: int, m: int, fmt: str = "mx",
                 mode: str = "sharq", tensor_scale: float | None = None, pairs: bool = False) -> dict:
    """Preparation for one path combination (reading R10).

    1. y = RMSNorm(x) * gamma (or y = x); for NVFP4 one S = amax(y)/2688;
    2. path 1 quantizes y (nothing when absent);
    3. R = y - D(path 1), in fp32;
    4. path 2 quantizes R (nothing when absent).
    Path 1's buffers are sp_codes / sp_meta / sp_scale, path 2's dn_codes /
    dn_meta / dn_scale; an absent path or a dense path's metadata has width 0.
    Mode "sharq" gives the buffers of prepare().
    """
    k1, k2 = MODE_PATHS[mode]
    x = bf16_bits_to_f32(x_bf16)
    T, K = x.shape
    g = None if gamma_bf16 is None else bf16_bits_to_f32(gamma_bf16)
    y, r = rmsnorm(x, g, eps)
    S = None
    if fmt == "nv":
        S = pts_scale(np.abs(y).max() if y.size else 0.0) if tensor_scale is None else np.float32(tensor_scale)
    elif fmt not in ("mx", "hif4"):
        raise ValueError(fmt)
    empty = np.zeros((T, 0), np.uint8)
    out = {"rows": T, "K": K, "n": n, "m": m, "pairs": pairs, "fmt": fmt, "mode": mode, "y": y, "r": r,
           "tensor_scale": None if S is None else np.float32(S)}
    p1 = quantize_path(y, k1, n, m, fmt, S, pairs) if k1 else None
    d1 = p1["deq"] if p1 else np.zeros(y.shape, np.float32)
    R = (y - d1).astype(np.float32)
    p2 = quantize_path(R, k2, n, m, fmt, S, pairs) if k2 else None
    d2 = p2["deq"] if p2 else np.zeros(y.shape, np.float32)
    out.update(sp_codes=p1["codes"] if p1 else empty, sp_meta=p1["meta"] if p1 else empty,
               sp_scale=p1["scale"] if p1 else empty, dn_codes=p2["codes"] if p2 else empty,
               dn_meta=p2["meta"] if p2 else empty, dn_scale=p2["scale"] if p2 else empty,
               keep=p1["keep"] if p1 else np.zeros(y.shape, bool),
               keep2=p2["keep"] if p2 else np.zeros(y.shape, bool), d_sp=d1, R=R, d_dn=d2)
    return out


def residual_add_bf16(x_bf16: np.ndarray, res_bf16: np.ndarray) -> np.ndarray:
    """h = bf16(x + res) (reading R9): the two bf16 values added in fp32 (IEEE,
    nearest even) and the fp32 sum rounded to bf16, nearest even.  Returns
    bf16 bit patterns."""
    s = (bf16_bits_to_f32(x_bf16) + bf16_bits_to_f32(res_bf16)).astype(np.float32)
    u = s.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def prepare_residual(x_bf16: np.ndarray, res_bf16: np.ndarray, gamma_bf16: np.ndarray | None, eps: float, n: int,
                     m: int, fmt: str = "mx", tensor_scale: float | None = None, pairs: bool = False) -> dict:
    """Preparation with the residual add in front of the RMSNorm: h = bf16(x + res)
    (R9), then prepare(h).  The dict also carries h (bf16 bits)."""
    h = residual_add_bf16(x_bf16, res_bf16)
    out = prepare(h, gamma_bf16, eps, n, m, fmt, tensor_scale, pairs)
    out["h"] = h
    return out


#: Cody-Waite split of ln 2 (R12): C1 carries the leading 16 bits of ln 2, so
#: k * C1 is exact for |k| < 2^8, and C2 = fl32(ln 2 - C1)
EXP_LN2_HI = np.float32(0.693145751953125)
EXP_LN2_LO = np.float32(1.428606765330187e-06)
EXP_LOG2E = np.float32(1.4426950408889634)
#: Taylor coefficients 1/j! (j = 7 .. 0) of e^r, rounded to fp32
EXP_TAYLOR = tuple(np.float32(1.0 / math.factorial(j)) for j in range(7, -1, -1))


def exp_nonpositive_f32(x: np.ndarray) -> np.ndarray:
    """e^x for fp32 x <= 0 by the recipe of reading R12, every step an IEEE
    fp32 operation rounded to nearest even (no fused multiply-add):
    Cody-Waite argument reduction x = k ln2 + r with k = rint(fl(x log2 e))
    and r = fl(fl(x - fl(k C1)) - fl(k C2)), the degree-7 Taylor polynomial of
    e^r in Horner form, then the exact power of two 2^k applied by one fp32
    multiply (which rounds into the subnormal range for k < -126).  Results
    below 2^-149 (k < -149) are 0."""
    x = np.asarray(x, dtype=np.float32)
    k = np.rint((x * EXP_LOG2E).astype(np.float32)).astype(np.float32)
    r = ((x - (k * EXP_LN2_HI).astype(np.float32)).astype(np.float32) - (k * EXP_LN2_LO).astype(np.float32))
    r = r.astype(np.float32)
    p = np.full(x.shape, EXP_TAYLOR[0], dtype=np.float32)
    for c in EXP_TAYLOR[1:]:
        p = ((p * r).astype(np.float32) + c).astype(np.float32)
    ki = k.astype(np.int64)
    two_k = pow2_f32(np.clip(ki, -149, 127))
    return np.where(ki < -149, np.float32(0.0), (p * two_k).astype(np.float32)).astype(np.float32)


def silu_mul_bf16(gate_bf16: np.ndarray, up_bf16: np.ndarray) -> np.ndarray:
    """Parity unpinned (reading R12: the recipe is a choice).
    h = bf16(SiLU(g) * u) by the fp32 recipe of reading R12: t = e^-|g|
    (exp_nonpositive_f32), q = fl(1 + t); s = fl(g / q) for g >= 0 and
    s = fl(fl(g t) / q) for g < 0 (SiLU(g) = g / (1 + e^-g) = g e^g / (1 + e^g)),
    with correctly rounded division; h = bf16(fl(s u)), nearest even.
    Returns bf16 bits."""
    g = bf16_bits_to_f32(gate_bf16)
    u = bf16_bits_to_f32(up_bf16)
    t = exp_nonpositive_f32(-np.abs(g))
    q = (np.float32(1.0) + t).astype(np.float32)
    num = np.where(g >= 0, g, (g * t).astype(np.float32)).astype(np.float32)
    sv = (num / q).astype(np.float32)
    with np.errstate(over="ignore"):
        h = (sv * u).astype(np.float32)
    return bf16_round_bits(h)


def bf16_round_bits(v: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, nearest with ties to even (finite inputs; overflow
    rounds to infinity as the fp32 -> bf16 conversion does)."""
    u = np.asarray(v, dtype=np.float32).view(np.uint32).astype(np.uint64)
    return ((u + 0x7FFF + ((u >> 16) & 1)) >> 16).astype(np.uint16)


def prepare_silu_mul(gate_bf16: np.ndarray, up_bf16: np.ndarray, n: int, m: int, fmt: str = "mx",
                     tensor_scale: float | None = None, pairs: bool = False) -> dict:
    """Preparation with SiLU.mul in front (R12), for the down projection (no
    RMSNorm): h = bf16(SiLU(g) * u), then prepare(h).  The dict also carries h."""
    h = silu_mul_bf16(gate_bf16, up_bf16)
    out = prepare(h, None, 0.0, n, m, fmt, tensor_scale, pairs)
    out["h"] = h
    return out


def quantize_weight(w_bf16: np.ndarray, fmt: str = "mx", scale_rule: str = "floor") -> dict:
    """Quantize W [N,K] once into one shared FP4 payload (Sec. 3.4, "Shared FP4 weights").

    MXFP4: E8M0 per 32 along K (rule "floor" or "ceil", R13), used by both
    paths.  NVFP4: per-tensor scale S_w = amax(W)/2688, E4M3 per 32 (the
    sparse view), and a dense view that repeats every scale for its two
    16-element halves.  HiF4: units of 64 along K with their three-level
    metadata, one view for both paths.
    """
    w = bf16_bits_to_f32(w_bf16)
    N, K = w.shape
    if scale_rule != "floor" and fmt != "mx":
        raise ValueError("the E8M0 scale rule applies to MXFP4 only")
    if fmt == "mx":
        c, _, s, deq = mx_quantize(w, None, scale_rule)
        return {"N": N, "K": K, "fmt": "mx", "codes": pack_nibbles(c), "scale": s,
                "scale_dn": s, "tensor_scale": None, "deq": deq}
    if fmt == "hif4":
        c, meta, deq = hif4_quantize(w)
        return {"N": N, "K": K, "fmt": "hif4", "codes": pack_nibbles(c), "scale": meta, "scale_dn": meta,
                "tensor_scale": None, "deq": deq}
    S = pts_scale(np.abs(w).max() if w.size else 0.0)
    c, _, s, deq = nv_quantize(w, S, MX_BLOCK)
    return {"N": N, "K": K, "fmt": "nv", "codes": pack_nibbles(c), "scale": s,
            "scale_dn": np.repeat(s, 2, axis=1), "tensor_scale": np.float32(S), "deq": deq}


# ---------------------------------------------------------------------------
# Dequantization from the packed buffers, and the two-path GEMM
# ---------------------------------------------------------------------------

def _block_scale_values(scale_codes: np.ndarray, fmt: str, block: int, K: int) -> np.ndarray:
    s = np.asarray(scale_codes)
    if fmt == "mx":
        vals = 2.0 ** (s.astype(np.float64) - 127.0)
    else:
        vals = e4m3_decode_bits(s)
    return np.repeat(vals, block, axis=1)[:, :K]


def _dequant_path(kind, codes, meta, scale, T: int, K: int, n: int, m: int, fmt: str, S: float) -> np.ndarray:
    if kind is None or (kind == "sparse" and n == 0):
        return np.zeros((T, K))
    if fmt == "hif4":
        dense = unpack_backbone(codes, meta, K, n, m)[0] if kind == "sparse" else unpack_nibbles(codes)
        return hif4_decode(dense, scale)
    if kind == "sparse":
        dense, keep = unpack_backbone(codes, meta, K, n, m)
        vals = e2m1_decode(dense) * _block_scale_values(scale, fmt, MX_BLOCK, K) * S
        return np.where(keep, vals, 0.0)
    block = MX_BLOCK if fmt == "mx" else NV_BLOCK
    return e2m1_decode(unpack_nibbles(codes)) * _block_scale_values(scale, fmt, block, K) * S


def dequant_act(act: dict):
    """Packed prepared activation -> (path 1 fp64 [T,K], path 2 fp64 [T,K]);
    for SharQ the backbone and the residual.  An absent path is zero.

    Values are exact: E2M1 x E8M0 (or x E4M3 x S) products fit in fp64.
    """
    K, n, m, fmt = act["K"], act["n"], act["m"], act["fmt"]
    T = act["rows"]
    k1, k2 = MODE_PATHS[act.get("mode", "sharq")]
    S = 1.0 if fmt != "nv" else float(act["tensor_scale"])
    a1 = _dequant_path(k1, act["sp_codes"], act["sp_meta"], act["sp_scale"], T, K, n, m, fmt, S)
    a2 = _dequant_path(k2, act["dn_codes"], act.get("dn_meta"), act["dn_scale"], T, K, n, m, fmt, S)
    return a1, a2


def _views(act: dict):
    """Weight scale view each path reads: the sparse view for a sparse path,
    the dense view for a dense one (Sec. 3.4)."""
    return tuple("sp" if k == "sparse" else "dn" for k in MODE_PATHS[act.get("mode", "sharq")])


def dequant_weight(wq: dict, view: str = "sp") -> np.ndarray:
    """Shared weight payload -> fp64 [N,K] through the sparse or the dense scale view."""
    K, fmt = wq["K"], wq["fmt"]
    if fmt == "hif4":
        return hif4_decode(unpack_nibbles(wq["codes"]), wq["scale"])
    S = 1.0 if fmt == "mx" else float(wq["tensor_scale"])
    if view == "sp" or fmt == "mx":
        sv = _block_scale_values(wq["scale"], fmt, MX_BLOCK, K)
    else:
        sv = _block_scale_values(wq["scale_dn"], fmt, NV_BLOCK, K)
    return e2m1_decode(unpack_nibbles(wq["codes"])) * sv * S


def linear(act: dict, wq: dict, rows: np.ndarray | None = None) -> np.ndarray:
    """Two-path output (eq. sharq-output) in fp64: Y = X~_sp W_sp^T + R~ W_dn^T;
    for the other modes the sum over their paths, each through its view.

    `rows` optionally restricts the computation to a subset of activation rows.
    """
    a1, a2 = dequant_act(act)
    if rows is not None:
        a1, a2 = a1[rows], a2[rows]
    v1, v2 = _views(act)
    return a1 @ dequant_weight(wq, v1).T + a2 @ dequant_weight(wq, v2).T


def linear_abs(act: dict, wq: dict, rows: np.ndarray | None = None) -> np.ndarray:
    """sum_k |a_1 w| + |a_2 w| per output: the scale of the accumulation error."""
    a1, a2 = dequant_act(act)
    if rows is not None:
        a1, a2 = a1[rows], a2[rows]
    v1, v2 = _views(act)
    return np.abs(a1) @ np.abs(dequant_weight(wq, v1)).T + np.abs(a2) @ np.abs(dequant_weight(wq, v2)).T


def linear_grouped(act: dict, row_index: np.ndarray | None, expert_offsets: np.ndarray,
                   weights: list) -> np.ndarray:
    """Grouped (MoE) form: Y[i] = SharQ(A[row_index[i]], W_e) for i in [off_e, off_e+1)."""
    total = int(expert_offsets[-1])
    N = weights[0]["N"]
    Y = np.zeros((total, N))
    a_sp, a_dn = dequant_act(act)
    for e, wq in enumerate(weights):
        lo, hi = int(expert_offsets[e]), int(expert_offsets[e + 1])
        if hi <= lo:
            continue
        rows = np.arange(lo, hi) if row_index is None else np.asarray(row_index[lo:hi])
        Y[lo:hi] = a_sp[rows] @ dequant_weight(wq, "sp").T + a_dn[rows] @ dequant_weight(wq, "dn").T
    return Y


def gemm_gate_error(y_hat: np.ndarray, y_ref: np.ndarray, y_abs: np.ndarray) -> float:
    """max |Y^ - Y| / sum_k(|a_sp w| + |a_dn w|), the componentwise accumulation error."""
    den = np.where(y_abs > 0, y_abs, 1.0)
    err = np.abs(np.asarray(y_hat, np.float64) - y_ref) / den
    err = np.where(y_abs > 0, err, np.abs(np.asarray(y_hat, np.float64) - y_ref))
    return float(err.max()) if err.size else 0.0


def subsets(m: int, n: int):
    """All n-subsets of range(m) (helper for brute-force checks)."""
    return itertools.combinations(range(m), n)


__all__ = [name for name in dir() if not name.startswith("_")] + ["_floor_log2_f32"]
