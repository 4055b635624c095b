// Device-side FP4 / block-scale helpers for gfx950 (CDNA4).
//
// E2M1 element codes: bit 3 sign, bits 0-2 index {0, .5, 1, 1.5, 2, 3, 4, 6}
// (SharQ App. A.1.2).  MXFP4 shares one E8M0 exponent per 32 values; NVFP4
// uses an E4M3 block scale plus a per-tensor fp32 scale (App. A.1.1-A.1.3).
//
// The hardware converter v_cvt_scalef32_pk_fp4_f32 rounds to the nearest E2M1
// value with ties to the even code, saturates at 6 and keeps the sign of zero;
// the kernels always hand it values already divided by the block scale and a
// unit scale operand, so the scale operand never has to represent 2^-127.
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

// OCP MX shared exponent of a block whose largest magnitude has bits
// `amax_bits`: floor(log2 amax) - 2, clamped at -127; -127 for an all-zero block.
__device__ __forceinline__ int mx_exponent(uint32_t amax_bits) {
  if (amax_bits == 0) return -127;
  int e = floor_log2_abs_bits(amax_bits) - 2;
  return e < -127 ? -127 : e;
}

// 2^-e as fp32 for e in [-127, 125]: always a normal number.
__device__ __forceinline__ float exp2_neg(int e) { return __uint_as_float((uint32_t)(127 - e) << 23); }

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

__device__ __forceinline__ float e4m3_value(uint32_t c) {
  uint32_t E = (c >> 3) & 15u, M = c & 7u;
  return E ? exp2_int((int)E - 7) * (1.0f + (float)M * 0.125f) : (float)M * 0.001953125f;
}

// Block quantizer policies.  enc(v) is the value handed to the E2M1
// converter (whose scale operand stays 1.0: the hardware uses only the
// exponent of that operand), dec(q) the dequantized value of a decoded code q.
//   MXFP4: power-of-two scale 2^e, both directions exact.
//   NVFP4: E4M3 block scale d under per-tensor scale S: enc = fl(v / fl(d S)),
//          dec = fl(fl(q d) S); a zero block scale gives signed-zero codes.
struct MxQ {
  float inv, sc;
  __device__ __forceinline__ float enc(float v) const { return v * inv; }
  __device__ __forceinline__ float dec(float q) const { return q * sc; }
};

struct NvQ {
  float d, step, S;
  __device__ __forceinline__ float enc(float v) const {
    if (!(d > 0.0f)) return v * 0.0f;   // keeps the sign of v
    return step > 0.0f ? v / step : v;
  }
  __device__ __forceinline__ float dec(float q) const { return (q * d) * S; }
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
  const float e0 = qz.enc(v[0]);
  // bytes 1-3 are written below, so the first conversion may start from any
  // register (e0's, which is dead after it)
  uint32_t t = __float_as_uint(e0);
  t = fp4x2<0>(t, e0, qz.enc(v[1]));
  t = fp4x2<1>(t, qz.enc(v[2]), qz.enc(v[3]));
  t = fp4x2<2>(t, qz.enc(v[4]), qz.enc(v[5]));
  t = fp4x2<3>(t, qz.enc(v[6]), qz.enc(v[7]));
  return t;
}

}  // namespace sharq
