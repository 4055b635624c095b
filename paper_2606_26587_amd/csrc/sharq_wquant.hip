// Weight preparation for SharQ on gfx950 (Sec. 3.4 "Shared FP4 weights with
// path-specific scales"; Fig. 2): W [N][K] is quantized once into one E2M1
// payload that both GEMM paths read.
//
// MXFP4: one lane per 32-value block along K; E8M0 exponent
// floor(log2 amax) - 2 (clamped at -127), codes E2M1(w / 2^e).  The payload
// and its scales are written panel-major (panels of 128 K positions, all N
// rows of a panel back to back), the layout the GEMM streams.  NVFP4 and
// HiF4 follow below.

#include "sharq_device.hpp"

#pragma clang fp contract(off)

namespace sharq {

template <typename T>
__device__ __forceinline__ void load32(const T* p, float (&v)[32]);

template <>
__device__ __forceinline__ void load32<uint16_t>(const uint16_t* p, float (&v)[32]) {
  const uint4* q = reinterpret_cast<const uint4*>(p);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint4 w = q[j];
    uint32_t u[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      v[8 * j + 2 * t] = bf16_lo(u[t]);
      v[8 * j + 2 * t + 1] = bf16_hi(u[t]);
    }
  }
}

template <>
__device__ __forceinline__ void load32<float>(const float* p, float (&v)[32]) {
  const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    float4 w = q[j];
    v[4 * j] = w.x; v[4 * j + 1] = w.y; v[4 * j + 2] = w.z; v[4 * j + 3] = w.w;
  }
}

template <typename T>
__global__ __launch_bounds__(256) void k_wquant_mx(const T* __restrict__ W, int N, int K, int64_t ldw,
                                                   uint8_t* __restrict__ codes, uint8_t* __restrict__ scale,
                                                   uint32_t rule_bias) {
  const int nblk = K / 32;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (int64_t)N * nblk) return;
  const int64_t n = gid / nblk;
  const int b = (int)(gid - n * nblk);
  float v[32];
  load32<T>(W + n * ldw + 32 * (int64_t)b, v);
  float amax = 0.0f;
#pragma unroll
  for (int k = 0; k < 32; ++k) amax = fmaxf(amax, fabsf(v[k]));
  const int e = mx_exponent(__float_as_uint(amax), rule_bias);
  const MxQ qz = MxQ::make(e);
  uint32_t q[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) q[w] = enc8(v + 8 * w, qz);
  // panel-major: panel p = b / 4 holds 128 K positions of all N rows
  const int p = b >> 2, j = b & 3, wp = min(128, K - 128 * p);
  const int64_t pn = (int64_t)p * N;
  *reinterpret_cast<uint4*>(codes + pn * 64 + n * (wp / 2) + 16 * j) = make_uint4(q[0], q[1], q[2], q[3]);
  scale[pn * 4 + n * (wp / 32) + j] = (uint8_t)(e + 127);
}

__device__ __forceinline__ float absmax32w(const float* v) {
  float m = 0.0f;
#pragma unroll
  for (int k = 0; k < 32; ++k) m = fmaxf(m, fabsf(v[k]));
  return m;
}

// NVFP4 weight (App. A.1.2-A.1.3; Fig. 2): per-tensor S_w = amax(W) / 2688,
// one E4M3 scale per 32 values (the sparse view), the dense view repeating it
// for both 16-value halves.  The running maximum is the bit pattern of a
// non-negative float in the tensor_scale slot, replaced by S_w afterwards.
// Blocks are walked grid-stride by at most kWAmaxWG workgroups, with one
// atomicMax per workgroup: atomics on one address serialize, and one per
// wavefront took ~0.4 ms on a 28672 x 4096 weight.
constexpr int kWAmaxWG = 1024;

template <typename T>
__global__ __launch_bounds__(256) void k_w_amax(const T* __restrict__ W, int N, int K, int64_t ldw, uint32_t* slot) {
  __shared__ float wmax[4];
  const int nblk = K / 32;
  const int64_t total = (int64_t)N * nblk;
  float m = 0.0f;
  for (int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x; gid < total; gid += (int64_t)gridDim.x * 256) {
    const int64_t n = gid / nblk;
    const int b = (int)(gid - n * nblk);
    float v[32];
    load32<T>(W + n * ldw + 32 * (int64_t)b, v);
    m = fmaxf(m, absmax32w(v));
  }
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) m = fmaxf(m, __shfl_xor(m, s, 64));
  if ((threadIdx.x & 63) == 0) wmax[threadIdx.x >> 6] = m;
  __syncthreads();
  if (threadIdx.x == 0) atomicMax(slot, __float_as_uint(fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]))));
}

__global__ void k_w_store_u32(uint32_t* p, uint32_t v) { *p = v; }

__global__ void k_w_pts_finalize(uint32_t* slot) {
  const float amax = __uint_as_float(*slot);
  *reinterpret_cast<float*>(slot) = amax > 0.0f ? amax / 2688.0f : 1.0f;
}

template <typename T>
__global__ __launch_bounds__(256) void k_wquant_nv(const T* __restrict__ W, int N, int K, int64_t ldw,
                                                   const float* S_ptr, uint8_t* __restrict__ codes,
                                                   uint8_t* __restrict__ scale, uint8_t* __restrict__ scale_dn) {
  const int nblk = K / 32;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (int64_t)N * nblk) return;
  const int64_t n = gid / nblk;
  const int b = (int)(gid - n * nblk);
  float v[32];
  load32<T>(W + n * ldw + 32 * (int64_t)b, v);
  const float S = *S_ptr;
  const NvQ q = NvQ::make(absmax32w(v), 6.0f * S, S);
  const int p = b >> 2, j = b & 3, wp = min(128, K - 128 * p);
  const int64_t pn = (int64_t)p * N;
  *reinterpret_cast<uint4*>(codes + pn * 64 + n * (wp / 2) + 16 * j) =
      make_uint4(enc8(v, q), enc8(v + 8, q), enc8(v + 16, q), enc8(v + 24, q));
  const uint8_t sb = (uint8_t)e4m3_bits(q.d);
  scale[pn * 4 + n * (wp / 32) + j] = sb;
  uint8_t* sd = scale_dn + pn * 8 + n * (wp / 16) + 2 * j;
  sd[0] = sb;
  sd[1] = sb;
}

// HiF4 weight: one thread per unit of 64 values along K (the conversion of
// the HiF4 appendix; see sharq_device.hpp).  Codes go to the unit's two
// 16-byte block slots, its 4 metadata bytes [E6M2, E1_8, E1_16 low, E1_16
// high] to the even block's 2-byte scale slots (one view for both paths).
template <typename T>
__global__ __launch_bounds__(256) void k_wquant_hif4(const T* __restrict__ W, int N, int K, int64_t ldw,
                                                     uint8_t* __restrict__ codes, uint8_t* __restrict__ scale) {
  const int nu = K / 64;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (gid >= (int64_t)N * nu) return;
  const int64_t n = gid / nu;
  const int u = (int)(gid - n * nu);
  float v[64];
  load32<T>(W + n * ldw + 64 * (int64_t)u, *reinterpret_cast<float(*)[32]>(v));
  load32<T>(W + n * ldw + 64 * (int64_t)u + 32, *reinterpret_cast<float(*)[32]>(v + 32));
  float v16[16], v8[8];
#pragma unroll
  for (int g = 0; g < 16; ++g)
    v16[g] = fmaxf(fmaxf(fabsf(v[4 * g]), fabsf(v[4 * g + 1])), fmaxf(fabsf(v[4 * g + 2]), fabsf(v[4 * g + 3])));
  float vmax = 0.0f;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    v8[i] = fmaxf(v16[2 * i], v16[2 * i + 1]);
    vmax = fmaxf(vmax, v8[i]);
  }
  const uint32_t code = e6m2_code(vmax * kOneSeventhBf16);
  const float rec = e6m2_rec(code);
  uint32_t e8 = 0u, e16 = 0u;
#pragma unroll
  for (int i = 0; i < 8; ++i) e8 |= (uint32_t)(v8[i] * rec >= 4.0f) << i;
#pragma unroll
  for (int g = 0; g < 16; ++g) e16 |= (uint32_t)(v16[g] * rec >= (((e8 >> (g >> 1)) & 1u) ? 4.0f : 2.0f)) << g;
  uint32_t q[8];
#pragma unroll
  for (int w = 0; w < 8; ++w) {
    uint32_t d = 0u;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int k = 8 * w + i;
      const int sh = (int)(((e8 >> (k >> 3)) & 1u) + ((e16 >> (k >> 2)) & 1u));
      d |= s1p2_code((v[k] * rec) * exp2_int(-sh)) << (4 * i);
    }
    q[w] = d;
  }
  const int b = 2 * u, p = b >> 2, j = b & 3, wp = min(128, K - 128 * p);
  const int64_t pn = (int64_t)p * N;
  uint4* c = reinterpret_cast<uint4*>(codes + pn * 64 + n * (wp / 2) + 16 * j);
  c[0] = make_uint4(q[0], q[1], q[2], q[3]);
  c[1] = make_uint4(q[4], q[5], q[6], q[7]);
  *reinterpret_cast<uint32_t*>(scale + (pn * 4 + n * (wp / 32) + j) * 2) =
      code | (e8 << 8) | (e16 << 16);
}

hipError_t launch_wquant_hif4(const void* W, int wdt, int N, int K, int64_t ldw, uint8_t* codes, uint8_t* scale,
                              hipStream_t st) {
  const int64_t total = (int64_t)N * (K / 64);
  dim3 grid((unsigned)((total + 255) / 256)), block(256);
  if (wdt == 2)
    k_wquant_hif4<float><<<grid, block, 0, st>>>(reinterpret_cast<const float*>(W), N, K, ldw, codes, scale);
  else
    k_wquant_hif4<uint16_t><<<grid, block, 0, st>>>(reinterpret_cast<const uint16_t*>(W), N, K, ldw, codes, scale);
  return hipGetLastError();
}

hipError_t launch_wquant_mx(const void* W, int wdt, int N, int K, int64_t ldw, uint8_t* codes, uint8_t* scale,
                            uint32_t rule_bias, hipStream_t st) {
  const int64_t total = (int64_t)N * (K / 32);
  dim3 grid((unsigned)((total + 255) / 256)), block(256);
  if (wdt == 2)
    k_wquant_mx<float><<<grid, block, 0, st>>>(reinterpret_cast<const float*>(W), N, K, ldw, codes, scale,
                                                rule_bias);
  else
    k_wquant_mx<uint16_t><<<grid, block, 0, st>>>(reinterpret_cast<const uint16_t*>(W), N, K, ldw, codes, scale,
                                                   rule_bias);
  return hipGetLastError();
}

hipError_t launch_wquant_nv(const void* W, int wdt, int N, int K, int64_t ldw, uint8_t* codes, uint8_t* scale,
                            uint8_t* scale_dn, float* ts, hipStream_t st) {
  const int64_t total = (int64_t)N * (K / 32);
  dim3 grid((unsigned)((total + 255) / 256)), block(256);
  uint32_t* slot = reinterpret_cast<uint32_t*>(ts);
  k_w_store_u32<<<1, 1, 0, st>>>(slot, 0u);
  const dim3 agrid(grid.x < (unsigned)kWAmaxWG ? grid.x : (unsigned)kWAmaxWG);
  if (wdt == 2) {
    k_w_amax<float><<<agrid, block, 0, st>>>(reinterpret_cast<const float*>(W), N, K, ldw, slot);
    k_w_pts_finalize<<<1, 1, 0, st>>>(slot);
    k_wquant_nv<float><<<grid, block, 0, st>>>(reinterpret_cast<const float*>(W), N, K, ldw, ts, codes, scale,
                                               scale_dn);
  } else {
    k_w_amax<uint16_t><<<agrid, block, 0, st>>>(reinterpret_cast<const uint16_t*>(W), N, K, ldw, slot);
    k_w_pts_finalize<<<1, 1, 0, st>>>(slot);
    k_wquant_nv<uint16_t><<<grid, block, 0, st>>>(reinterpret_cast<const uint16_t*>(W), N, K, ldw, ts, codes,
                                                  scale, scale_dn);
  }
  return hipGetLastError();
}

}  // namespace sharq
