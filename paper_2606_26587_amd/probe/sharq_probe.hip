// Sustained scaled-FP4 MFMA rate and shader clock (a measurement aid for the
// benchmark; not part of the method).  Every wavefront keeps 8 independent
// 32x32 accumulators in flight and cycles its operands through four register
// sets of pseudo-random E2M1 codes, so consecutive MFMAs never wait on each
// other and the operand data keeps changing like a real GEMM's.

#include <hip/hip_runtime.h>
#include <cstdint>

#include "sharq_probe.h"

namespace {

typedef float v16f __attribute__((ext_vector_type(16)));
typedef int v8i __attribute__((ext_vector_type(8)));

__device__ __forceinline__ uint32_t hash32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x7feb352du;
  h ^= h >> 15;
  h *= 0x846ca68bu;
  h ^= h >> 16;
  return h;
}

__global__ __launch_bounds__(256, 1) void k_mfma_fp4_rate(float* sink, unsigned long long* clk, int iters) {
  const uint32_t g = blockIdx.x * 256u + threadIdx.x;
  v8i a[4], b[4];
#pragma unroll
  for (int j = 0; j < 4; ++j)
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      a[j][i] = (int)hash32(g * 64u + j * 8u + i);
      b[j][i] = (int)hash32(0x9E3779B9u ^ (g * 64u + j * 8u + i));
    }
  v16f acc[8];
#pragma unroll
  for (int f = 0; f < 8; ++f)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[f][r] = 0.0f;
  const uint64_t t0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int f = 0; f < 8; ++f)   // E2M1 x E2M1 (format 4), E8M0 scale 127 = 1.0
        acc[f] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a[j], b[(j + f) & 3], acc[f], 4, 4, 0, 127, 0, 127);
  }
  const uint64_t t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.0f;
#pragma unroll
  for (int f = 0; f < 8; ++f)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[f][r];
  sink[g] = s;
  if (threadIdx.x == 0) {
    clk[2 * blockIdx.x] = t1 - t0;
    clk[2 * blockIdx.x + 1] = r1 - r0;
  }
}

// The same for the 16-bit MFMAs (v_mfma_f32_32x32x16_bf16 / _f16), which the
// NVFP4 and HiF4 GEMMs run on: pseudo-random finite operands (sign, exponent
// 2^-7..2^8, random mantissa), four sets cycled, 8 accumulators.
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

template <typename V, typename E>
__device__ __forceinline__ V operand16(uint32_t seed) {
  V v;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const uint32_t h = hash32(seed * 8u + (uint32_t)i);
    const float x = __uint_as_float((h & 0x807FFFFFu) | ((120u + ((h >> 23) & 15u)) << 23));
    v[i] = (E)x;
  }
  return v;
}

__device__ __forceinline__ v16f mfma16(bf16x8 a, bf16x8 b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v16f mfma16(f16x8 a, f16x8 b, v16f c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
}

template <typename V, typename E>
__global__ __launch_bounds__(256, 1) void k_mfma16_rate(float* sink, unsigned long long* clk, int iters) {
  const uint32_t g = blockIdx.x * 256u + threadIdx.x;
  V a[4], b[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    a[j] = operand16<V, E>(g * 8u + (uint32_t)j);
    b[j] = operand16<V, E>(0x9E3779B9u ^ (g * 8u + (uint32_t)j));
  }
  v16f acc[8];
#pragma unroll
  for (int f = 0; f < 8; ++f)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[f][r] = 0.0f;
  const uint64_t t0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int f = 0; f < 8; ++f) acc[f] = mfma16(a[j], b[(j + f) & 3], acc[f]);
  }
  const uint64_t t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
  float s = 0.0f;
#pragma unroll
  for (int f = 0; f < 8; ++f)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += acc[f][r];
  sink[g] = s;
  if (threadIdx.x == 0) {
    clk[2 * blockIdx.x] = t1 - t0;
    clk[2 * blockIdx.x + 1] = r1 - r0;
  }
}

}  // namespace

extern "C" __attribute__((visibility("default"))) int sharq_probe_mfma_bf16(int iters, int workgroups, float* sink,
                                                                            unsigned long long* clk,
                                                                            hipStream_t stream) {
  if (iters < 1 || workgroups < 1 || sink == nullptr || clk == nullptr) return (int)hipErrorInvalidValue;
  k_mfma16_rate<bf16x8, __bf16><<<dim3((unsigned)workgroups), dim3(256), 0, stream>>>(sink, clk, iters);
  return (int)hipGetLastError();
}

extern "C" __attribute__((visibility("default"))) int sharq_probe_mfma_f16(int iters, int workgroups, float* sink,
                                                                           unsigned long long* clk,
                                                                           hipStream_t stream) {
  if (iters < 1 || workgroups < 1 || sink == nullptr || clk == nullptr) return (int)hipErrorInvalidValue;
  k_mfma16_rate<f16x8, _Float16><<<dim3((unsigned)workgroups), dim3(256), 0, stream>>>(sink, clk, iters);
  return (int)hipGetLastError();
}

extern "C" __attribute__((visibility("default"))) int sharq_probe_mfma_fp4(int iters, int workgroups, float* sink,
                                                                           unsigned long long* clk,
                                                                           hipStream_t stream) {
  if (iters < 1 || workgroups < 1 || sink == nullptr || clk == nullptr) return (int)hipErrorInvalidValue;
  k_mfma_fp4_rate<<<dim3((unsigned)workgroups), dim3(256), 0, stream>>>(sink, clk, iters);
  return (int)hipGetLastError();
}
