// Device-side FP4 / block-scale helpers for gfx950 (CDNA4).
//
// E2M1 element codes: bit 3 sign, bits 0-2 index {0, .5, 1, 1.5, 2, 3, 4, 6}
// (SharQ App. A.1.2).  MXFP4 shares one E8M0 exponent per 32 values; NVFP4
// uses an E4M3 block scale plus a per-tensor fp32 scale (App. A.1.1-A.1.3).
//
// The hardware converter v_cvt_scalef32_pk_fp4_f32 rounds to the nearest E2M1
// value with ties to the even code, saturates at 6 and keeps the sign of zero.
// MXFP4 blocks hand it their power-of-two scale through its scale operand;
// NVFP4 blocks hand it values already divided by their scale, with a unit
// scale operand.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sharq {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// floor(log2 a) for a > 0, from the bits of |a| (normal or subnormal).
__device__ __forceinline__ int floor_log2_abs_bits(uint32_t abits) {
  uint32_t ex = abits >> 23;
  return ex ? (int)ex - 127 : (31 - (int)__builtin_clz(abits)) - 149;
}

// E8M0 rules of the shared exponent of a block whose largest magnitude has
// bits `amax_bits` (non-negative, finite), as the bias added to those bits:
//   kE8Floor  floor(log2 amax) - 2 (OCP MX): the exponent field minus 129;
//   kE8Ceil   ceil(log2(amax / 6)), the smallest power of two under which the
//             peak does not exceed 6: one more than the floor rule exactly
//             when the mantissa is above 1.5 (6 * 2^(E-2) = 1.5 * 2^E), i.e.
//             when adding 0x3FFFFF carries into the exponent field.
// Both clamped at -127; subnormal and zero maxima give -127.
constexpr uint32_t kE8Floor = 0u, kE8Ceil = 0x3FFFFFu;

__device__ __forceinline__ int mx_exponent(uint32_t amax_bits, uint32_t rule_bias = kE8Floor) {
  const int e = (int)((amax_bits + rule_bias) >> 23) - 129;
  return e < -127 ? -127 : e;
}

// Options of a preparation beyond its buffers: the E8M0 rule (MXFP4) and
// the optional debug outputs (keep bits per block, RMSNorm r per row).
struct PrepExtras {
  uint32_t rule_bias;
  uint32_t* dbg_mask;
  float* dbg_r;
};

// 2^e as fp32 for e in [-149, 127] (2^-127 is subnormal).
__device__ __forceinline__ float exp2_int(int e) {
  return e >= -126 ? __uint_as_float((uint32_t)(e + 127) << 23) : __uint_as_float(1u << (e + 149));
}

// Two fp32 values (already divided by their block scale) -> two E2M1 codes in
// byte SEL of `old` (first value in the low nibble).
template <int SEL>
__device__ __forceinline__ uint32_t fp4x2(uint32_t old, float a, float b) {
  return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, 1.0f, SEL);
}

// Byte SEL of `packed` (two E2M1 codes) -> their two values (low nibble first).
template <int SEL>
__device__ __forceinline__ v2f fp4x2_decode(uint32_t packed) {
  return __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(packed, 1.0f, SEL);
}

__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Round a non-negative fp32 value to E4M3 (bias 7, max 448, subnormal step
// 2^-9), nearest with ties to even, saturating.  Returns the rounded value.
__device__ __forceinline__ float e4m3_round(float a) {
  if (!(a > 0.0f)) return 0.0f;
  if (a >= 448.0f) return 448.0f;
  uint32_t b = __float_as_uint(a);
  int E = floor_log2_abs_bits(b);
  if (E < -6) E = -6;
  // quantum 2^(E-3); scale a to units of the quantum (exact), round half even
  float q_inv = exp2_int(3 - E);
  float t = a * q_inv;                     // exact: power-of-two scaling of a normal value
  float r = __builtin_rintf(t);            // round half to even
  float out = r * exp2_int(E - 3);         // exact
  return out > 448.0f ? 448.0f : out;
}

// E4M3 value (non-negative, representable) -> 8-bit code.
__device__ __forceinline__ uint32_t e4m3_bits(float v) {
  if (!(v > 0.0f)) return 0u;
  uint32_t b = __float_as_uint(v);
  int E = floor_log2_abs_bits(b);
  if (E >= -6) {
    uint32_t man = (b >> 20) & 7u;         // top 3 mantissa bits (value is representable)
    return ((uint32_t)(E + 7) << 3) | man;
  }
  return (uint32_t)__builtin_rintf(v * 512.0f);   // subnormal: v = m * 2^-9
}

// The value of an E4M3 scale code (bias 7, largest finite 448, the sign bit
// ignored).  gfx950's FP8 conversion decodes this E4M3 exactly: checked on
// the GPU against the format's definition for all 256 codes, subnormals
// included.  It differs from the definition only for code 0x7F (NaN there),
// which no scale takes: scales saturate at 448 = 0x7E.
__device__ __forceinline__ float e4m3_value(uint32_t c) {
  return __builtin_amdgcn_cvt_f32_fp8((int)(c & 0x7Fu), 0);
}

// Block quantizer policies.  enc2<SEL>(old, a, b) writes the E2M1 codes of
// two values into byte SEL of `old` (first value in the low nibble);
// dec2<SEL>(packed) returns the dequantized values of the two codes in byte
// SEL.
//   MXFP4: power-of-two block scale 2^e.  The converters divide (encode) or
//          multiply (decode) by 2^k, k the exponent field of their scale
//          operand minus 127 (checked on gfx950 for every k in [-127, 127],
//          subnormal values included), so the block exponent goes straight
//          into that operand: a float with exponent field e + 127, which is
//          the bit pattern of 0.0f for e = -127.  Both directions are exact.
//   NVFP4: E4M3 block scale d under per-tensor scale S: the converter gets
//          fl(v / fl(d S)) with a unit scale, dec = fl(fl(q d) S); a zero
//          block scale gives signed-zero codes.
struct MxQ {
  float sc;
  __device__ static MxQ make(int e) {
    MxQ q;
    q.sc = __uint_as_float((uint32_t)(e + 127) << 23);
    return q;
  }
  template <int SEL>
  __device__ __forceinline__ uint32_t enc2(uint32_t old, float a, float b) const {
    return __builtin_amdgcn_cvt_scalef32_pk_fp4_f32(old, a, b, sc, SEL);
  }
  template <int SEL>
  __device__ __forceinline__ v2f dec2(uint32_t packed) const {
    return __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(packed, sc, SEL);
  }
};

struct NvQ {
  float d, step, S;
  __device__ __forceinline__ float enc(float v) const {
    if (!(d > 0.0f)) return v * 0.0f;   // keeps the sign of v
    return step > 0.0f ? v / step : v;
  }
  __device__ __forceinline__ float dec(float q) const { return (q * d) * S; }
  template <int SEL>
  __device__ __forceinline__ uint32_t enc2(uint32_t old, float a, float b) const {
    return fp4x2<SEL>(old, enc(a), enc(b));
  }
  template <int SEL>
  __device__ __forceinline__ v2f dec2(uint32_t packed) const {
    const v2f q = fp4x2_decode<SEL>(packed);
    v2f r;
    r.x = dec(q.x);
    r.y = dec(q.y);
    return r;
  }
  __device__ static NvQ make(float amax, float six_s, float S) {
    NvQ q;
    q.d = e4m3_round(amax / six_s);
    q.step = q.d * S;
    q.S = S;
    return q;
  }
};

// Eight consecutive values -> one dword of E2M1 codes under quantizer qz.
template <class Q>
__device__ __forceinline__ uint32_t enc8(const float* v, const Q& qz) {
  // bytes 1-3 are written below, so the first conversion may start from any
  // register (v[0]'s)
  uint32_t t = __float_as_uint(v[0]);
  t = qz.template enc2<0>(t, v[0], v[1]);
  t = qz.template enc2<1>(t, v[2], v[3]);
  t = qz.template enc2<2>(t, v[4], v[5]);
  t = qz.template enc2<3>(t, v[6], v[7]);
  return t;
}

// ---------------------------------------------------------------------------
// Backbone expansion: compressed 32-position block -> 32 dense E2M1 nibbles
// ---------------------------------------------------------------------------

// One output dword (8 K positions) of an expanded block.
// 2:4: byte g of `c` holds group g's two kept codes (lower K first); nibble g
// of `meta` holds their positions i0 | i1 << 2.  Dword D covers groups 2D, 2D+1.
// 4:8: bytes 2g, 2g+1 of `c` hold group g's four kept codes (ascending K);
// byte g of `meta` is its keep mask.  Dword D is group D.
template <int PAT, int D>
__device__ __forceinline__ uint32_t expand_dw(uint2 c, uint32_t meta) {
  const uint32_t cw = D < 2 ? c.x : c.y;
  uint32_t r = 0u;
  if (PAT == 24) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int g = 2 * D + h;
      const uint32_t byte = (cw >> (8 * (g & 3))) & 0xFFu;
      const uint32_t nib = (meta >> (4 * g)) & 0xFu;
      r |= (byte & 0xFu) << (4 * (nib & 3u) + 16 * h);
      r |= (byte >> 4) << (4 * (nib >> 2) + 16 * h);
    }
  } else {
    uint32_t c16 = (cw >> (16 * (D & 1))) & 0xFFFFu;
    const uint32_t mask = (meta >> (8 * D)) & 0xFFu;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      if ((mask >> p) & 1u) {
        r |= (c16 & 0xFu) << (4 * p);
        c16 >>= 4;
      }
    }
  }
  return r;
}

// A compressed 32-position block -> 32 dense E2M1 nibbles.
template <int PAT>
__device__ __forceinline__ uint4 expand_block(uint2 c, uint32_t meta) {
  return make_uint4(expand_dw<PAT, 0>(c, meta), expand_dw<PAT, 1>(c, meta), expand_dw<PAT, 2>(c, meta),
                    expand_dw<PAT, 3>(c, meta));
}

// ---------------------------------------------------------------------------
// HiF4 (a three-level scaled 4-bit format; App. "HiFloat4 (HiF4) Data
// Format"): units of 64 values along K; an E6M2 level-1 scale (6 exponent
// bits, bias 48, 2 mantissa bits, normal values only, all-ones = NaN), one
// micro-exponent bit per 8 values (E1_8) and per 4 values (E1_16), S1P2
// elements (sign, magnitude m in {0..7}, value m/4).  V = E6M2 *
// 2^(E1_8 + E1_16) * S1P2 (eq. "hif4-value").  The conversion follows the
// paper's algorithm on fp32 inputs: SF = fl(Vmax * bf16(1/7)), E6M2 = SF to
// 2 mantissa bits (nearest even, clamped to [2^-48, 1.5 * 2^15]),
// REC = bf16(1/1.M) * 2^-E, E1_8 = (V8 * REC >= 4), E1_16 = (V16 * REC >=
// 2^(1 + E1_8)), scaled = fl(v * REC) * 2^-(E1_8 + E1_16), S1P2 = nearest
// quarter, ties to even, saturating at 1.75.
// ---------------------------------------------------------------------------

constexpr float kOneSeventhBf16 = 0.142578125f;   // bf16(1/7)

__device__ __forceinline__ uint32_t e6m2_code(float sf) {
  if (!(sf >= 0x1p-48f)) return 0u;   // below the smallest normal (zero included)
  const uint32_t b = __float_as_uint(sf);
  int E = (int)(b >> 23) - 127;
  const uint32_t mant = b & 0x7FFFFFu;
  uint32_t q = mant >> 21;
  const uint32_t rest = mant & 0x1FFFFFu;
  if (rest > 0x100000u || (rest == 0x100000u && (q & 1u))) ++q;
  if (q == 4u) {
    q = 0u;
    ++E;
  }
  if (E > 15 || (E == 15 && q == 3u)) return 0xFEu;   // largest finite: 1.5 * 2^15
  return ((uint32_t)(E + 48) << 2) | q;
}

__device__ __forceinline__ float e6m2_value(uint32_t code) {
  return exp2_int((int)(code >> 2) - 48) * (1.0f + 0.25f * (float)(code & 3u));
}

// bf16(1/1.M) * 2^-E: the reciprocal table of the conversion algorithm
__device__ __forceinline__ float e6m2_rec(uint32_t code) {
  const uint32_t M = code & 3u;
  const float t = M == 0 ? 1.0f : M == 1 ? 0.80078125f : M == 2 ? 0.66796875f : 0.5703125f;
  return t * exp2_int(48 - (int)(code >> 2));
}

// scaled fp32 value -> S1P2 code (bit 3 sign, bits 0-2 magnitude)
__device__ __forceinline__ uint32_t s1p2_code(float s) {
  const float m = fminf(__builtin_rintf(fabsf(s) * 4.0f), 7.0f);
  return ((__float_as_uint(s) >> 28) & 8u) | (uint32_t)m;
}

// S1P2 code times a (power-of-two multiple of the) level-1 scale
__device__ __forceinline__ float s1p2_value(uint32_t c, float scale) {
  const float v = (float)(c & 7u) * 0.25f * scale;
  return (c & 8u) ? -v : v;
}

}  // namespace sharq
