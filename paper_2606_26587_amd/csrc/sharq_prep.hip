// Fused SharQ activation preparation for gfx950 (SharQ Sec. 3.4, "Fused
// sparse-residual preparation"; Fig. 2).
//
// One wavefront per activation row.  Lane l owns whole 32-element blocks
// b = l, l + 64, l + 128, ... of its row, so every block-local step (N:M
// selection inside groups of 4 or 8, the block max behind each scale, the
// residual) runs inside one lane without cross-lane traffic; only the RMSNorm
// sum of squares crosses lanes.  Every row is read from HBM once and every
// output byte is written once.
//
// Per block of 32 normalized values y (eq. numbers of Sec. 3.3):
//   mask     keep the n largest |y| of each group of m, ties to the lower index
//            ("dynamic-mask" / "sharq-sparse-backbone");
//   backbone E8M0 scale from the block max of the kept values, E2M1 codes of
//            the kept values, compressed with index metadata
//            ("sharq-quantized-backbone");
//   residual R = y - dequant(backbone) in fp32, exact for MXFP4
//            ("sharq-residual"), then its own E8M0 scale and E2M1 codes.
//
// The RMSNorm sum of squares is evaluated as a balanced binary tree over the
// row padded with zeros to a power of two: the 32 squares of a block pairwise
// inside the lane, then an xor butterfly over the 64 lanes (a 2048-element
// chunk), then the chunks pairwise.  This fixes the fp32 result independently
// of the launch shape.

#include "sharq_device.hpp"

#pragma clang fp contract(off)

namespace sharq {

// ---------------------------------------------------------------------------
// N:M selection inside one block
// ---------------------------------------------------------------------------

// 2:4 on one group: keep bits of positions 0..3 (exactly two set).
__device__ __forceinline__ void top2of4(float y0, float y1, float y2, float y3, bool& k0, bool& k1,
                                        bool& k2, bool& k3) {
  float a0 = fabsf(y0), a1 = fabsf(y1), a2 = fabsf(y2), a3 = fabsf(y3);
  // cij: position i wins against position j (i < j; a tie goes to i)
  int c01 = a0 >= a1, c02 = a0 >= a2, c03 = a0 >= a3;
  int c12 = a1 >= a2, c13 = a1 >= a3, c23 = a2 >= a3;
  // position p is kept iff it wins at least 2 of its 3 comparisons
  k0 = (c01 + c02 + c03) >= 2;
  k1 = ((1 - c01) + c12 + c13) >= 2;
  k2 = ((1 - c02) + (1 - c12) + c23) >= 2;
  k3 = ((1 - c03) + (1 - c13) + (1 - c23)) >= 2;
}

template <int SEL>
__device__ __forceinline__ void put_pair(uint32_t& word, float a, float b) {
  word = fp4x2<SEL>(word, a, b);
}

__device__ __forceinline__ void put_pair_dyn(uint32_t& word, int sel, float a, float b) {
  switch (sel & 3) {
    case 0: put_pair<0>(word, a, b); break;
    case 1: put_pair<1>(word, a, b); break;
    case 2: put_pair<2>(word, a, b); break;
    default: put_pair<3>(word, a, b); break;
  }
}

__device__ __forceinline__ v2f get_pair_dyn(uint32_t word, int sel) {
  switch (sel & 3) {
    case 0: return fp4x2_decode<0>(word);
    case 1: return fp4x2_decode<1>(word);
    case 2: return fp4x2_decode<2>(word);
    default: return fp4x2_decode<3>(word);
  }
}

// Backbone of one block for the 2:4 pattern.  Returns the residual in R.
__device__ __forceinline__ void backbone_24(const float (&y)[32], float inv, float sc, uint32_t (&codes)[2],
                                            uint32_t& meta, float (&R)[32]) {
  codes[0] = codes[1] = 0u;
  meta = 0u;
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    float y0 = y[4 * g], y1 = y[4 * g + 1], y2 = y[4 * g + 2], y3 = y[4 * g + 3];
    bool k0, k1, k2, k3;
    top2of4(y0, y1, y2, y3, k0, k1, k2, k3);
    float v0 = k0 ? y0 : (k1 ? y1 : y2);            // first kept (ascending K)
    float v1 = k3 ? y3 : (k2 ? y2 : y1);            // second kept
    uint32_t i0 = k0 ? 0u : (k1 ? 1u : 2u);
    uint32_t i1 = k3 ? 3u : (k2 ? 2u : 1u);
    meta |= (i0 | (i1 << 2)) << (4 * g);
    put_pair_dyn(codes[g >> 2], g, v0 * inv, v1 * inv);
    v2f d = get_pair_dyn(codes[g >> 2], g);
    float d0 = d.x * sc, d1 = d.y * sc;            // exact: power-of-two scale
    R[4 * g + 0] = y0 - (k0 ? d0 : 0.0f);
    R[4 * g + 1] = y1 - (k1 ? (k0 ? d1 : d0) : 0.0f);
    R[4 * g + 2] = y2 - (k2 ? (k3 ? d0 : d1) : 0.0f);
    R[4 * g + 3] = y3 - (k3 ? d1 : 0.0f);
  }
}

// Backbone of one block for the 4:8 pattern (keep mask metadata).
__device__ __forceinline__ void backbone_48(const float (&y)[32], float inv, float sc, uint32_t (&codes)[2],
                                            uint32_t& meta, float (&R)[32]) {
  codes[0] = codes[1] = 0u;
  meta = 0u;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    float a[8];
#pragma unroll
    for (int p = 0; p < 8; ++p) a[p] = fabsf(y[8 * g + p]);
    bool keep[8];
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      int rank = 0;
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        if (q < p) rank += a[q] >= a[p];
        if (q > p) rank += a[q] > a[p];
      }
      keep[p] = rank < 4;
    }
    // kept values in ascending position order
    float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    int pre[8];
    int cnt = 0;
    uint32_t mask = 0u;
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      pre[p] = cnt;
#pragma unroll
      for (int s = 0; s < 4; ++s)
        if (keep[p] && cnt == s) v[s] = y[8 * g + p];
      cnt += keep[p];
      mask |= (uint32_t)keep[p] << p;
    }
    meta |= mask << (8 * g);
    int byte0 = 2 * g;   // group g's four codes occupy bytes 2g, 2g+1 of the 8
    put_pair_dyn(codes[byte0 >> 2], byte0, v[0] * inv, v[1] * inv);
    put_pair_dyn(codes[(byte0 + 1) >> 2], byte0 + 1, v[2] * inv, v[3] * inv);
    v2f d01 = get_pair_dyn(codes[byte0 >> 2], byte0);
    v2f d23 = get_pair_dyn(codes[(byte0 + 1) >> 2], byte0 + 1);
    float d[4] = {d01.x * sc, d01.y * sc, d23.x * sc, d23.y * sc};
#pragma unroll
    for (int p = 0; p < 8; ++p) {
      float dp = 0.0f;
#pragma unroll
      for (int s = 0; s < 4; ++s)
        if (keep[p] && pre[p] == s) dp = d[s];
      R[8 * g + p] = y[8 * g + p] - dp;
    }
  }
}

// Quantize and store one block: backbone + residual.
template <int PAT>
__device__ __forceinline__ void block_mx(const float (&y)[32], uint8_t* __restrict__ spc, uint8_t* __restrict__ spm,
                                         uint8_t* __restrict__ sps, uint8_t* __restrict__ dnc,
                                         uint8_t* __restrict__ dns) {
  // The group maximum is always kept, so the backbone block max equals the
  // block max of y.
  float amax = 0.0f;
#pragma unroll
  for (int k = 0; k < 32; ++k) amax = fmaxf(amax, fabsf(y[k]));
  int e = mx_exponent(__float_as_uint(amax));
  float inv = exp2_neg(e), sc = exp2_int(e);
  uint32_t codes[2], meta;
  float R[32];
  if (PAT == 24)
    backbone_24(y, inv, sc, codes, meta, R);
  else
    backbone_48(y, inv, sc, codes, meta, R);

  float ramax = 0.0f;
#pragma unroll
  for (int k = 0; k < 32; ++k) ramax = fmaxf(ramax, fabsf(R[k]));
  int er = mx_exponent(__float_as_uint(ramax));
  float rinv = exp2_neg(er);
  uint32_t dn[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    uint32_t t = 0u;
    t = fp4x2<0>(t, R[8 * w + 0] * rinv, R[8 * w + 1] * rinv);
    t = fp4x2<1>(t, R[8 * w + 2] * rinv, R[8 * w + 3] * rinv);
    t = fp4x2<2>(t, R[8 * w + 4] * rinv, R[8 * w + 5] * rinv);
    t = fp4x2<3>(t, R[8 * w + 6] * rinv, R[8 * w + 7] * rinv);
    dn[w] = t;
  }
  *reinterpret_cast<uint2*>(spc) = make_uint2(codes[0], codes[1]);
  *reinterpret_cast<uint32_t*>(spm) = meta;
  *sps = (uint8_t)(e + 127);
  *reinterpret_cast<uint4*>(dnc) = make_uint4(dn[0], dn[1], dn[2], dn[3]);
  *dns = (uint8_t)(er + 127);
}

__device__ __forceinline__ void unpack_bf16x32(const uint4 (&q)[4], float (&x)[32]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t w[4] = {q[j].x, q[j].y, q[j].z, q[j].w};
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      x[8 * j + 2 * t] = bf16_lo(w[t]);
      x[8 * j + 2 * t + 1] = bf16_hi(w[t]);
    }
  }
}

// Balanced-tree sum of the 32 squares of one block.
__device__ __forceinline__ float block_sum_sq(const float (&x)[32]) {
  float s[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) s[k] = x[2 * k] * x[2 * k] + x[2 * k + 1] * x[2 * k + 1];
#pragma unroll
  for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
    for (int k = 0; k < w; ++k) s[k] = s[2 * k] + s[2 * k + 1];
  return s[0];
}

__device__ __forceinline__ float wave_tree_sum(float v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v = v + __shfl_xor(v, m, 64);
  return v;
}

// Output addressing.  Every buffer is panel-major: K is cut into panels of
// 128 positions (4 scale blocks; the last panel may be narrower) and panel p
// stores the bytes of all M rows for its K range, row after row.  Block b of
// a row is block j = b % 4 of panel p = b / 4.
struct ActOut {
  uint8_t *spc, *spm, *sps, *dnc, *dns;
  int64_t M;
  int K;
};

struct BlockOut {
  uint8_t *spc, *spm, *sps, *dnc, *dns;
};

__device__ __forceinline__ BlockOut block_out(const ActOut& o, int64_t row, int b) {
  const int p = b >> 2, j = b & 3;
  const int wp = min(128, o.K - 128 * p);   // panel width in K positions
  const int64_t pm = (int64_t)p * o.M;
  BlockOut r;
  r.dnc = o.dnc + pm * 64 + row * (wp / 2) + 16 * j;
  r.spc = o.spc + pm * 32 + row * (wp / 4) + 8 * j;
  r.spm = o.spm + pm * 16 + row * (wp / 8) + 4 * j;
  r.sps = o.sps + pm * 4 + row * (wp / 32) + j;
  r.dns = o.dns + pm * 4 + row * (wp / 32) + j;
  return r;
}

// RMSNorm variant: the row's blocks stay in registers between the sum of
// squares and the quantization.  NB = blocks per lane, a power of two.
template <int NB, int PAT>
__global__ __launch_bounds__(256) void k_prep_mx_norm(const uint16_t* __restrict__ X, int M, int K, int64_t ldx,
                                                      const uint16_t* __restrict__ gamma, float eps,
                                                      uint8_t* sp_codes, uint8_t* sp_meta, uint8_t* sp_scale,
                                                      uint8_t* dn_codes, uint8_t* dn_scale) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;   // whole wavefront; the kernel has no block barrier
  const int nblk = K / 32;
  const uint4* xr = reinterpret_cast<const uint4*>(X + row * ldx);
  uint4 xs[NB][4];
  float chunk[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int b = lane + 64 * i;
    if (b < nblk) {
#pragma unroll
      for (int j = 0; j < 4; ++j) xs[i][j] = xr[4 * b + j];
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j) xs[i][j] = make_uint4(0u, 0u, 0u, 0u);
    }
  }
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    float x[32];
    unpack_bf16x32(xs[i], x);
    chunk[i] = wave_tree_sum(block_sum_sq(x));
  }
#pragma unroll
  for (int w = NB / 2; w >= 1; w >>= 1)
#pragma unroll
    for (int k = 0; k < w; ++k) chunk[k] = chunk[2 * k] + chunk[2 * k + 1];
  const float r = (float)(1.0 / __builtin_sqrt((double)chunk[0] / (double)K + (double)eps));

  const ActOut o{sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, (int64_t)M, K};
  const uint4* gr = reinterpret_cast<const uint4*>(gamma);
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int b = lane + 64 * i;
    if (b >= nblk) break;
    uint4 gq[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) gq[j] = gr[4 * b + j];
    float x[32], g[32], y[32];
    unpack_bf16x32(xs[i], x);
    unpack_bf16x32(gq, g);
#pragma unroll
    for (int k = 0; k < 32; ++k) {
      float t = x[k] * r;
      y[k] = t * g[k];
    }
    const BlockOut d = block_out(o, row, b);
    block_mx<PAT>(y, d.spc, d.spm, d.sps, d.dnc, d.dns);
  }
}

// Variant without RMSNorm: a plain stream over the row's blocks.
template <int PAT>
__global__ __launch_bounds__(256) void k_prep_mx_plain(const uint16_t* __restrict__ X, int M, int K, int64_t ldx,
                                                       uint8_t* sp_codes, uint8_t* sp_meta, uint8_t* sp_scale,
                                                       uint8_t* dn_codes, uint8_t* dn_scale) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;
  const int nblk = K / 32;
  const uint4* xr = reinterpret_cast<const uint4*>(X + row * ldx);
  const ActOut o{sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, (int64_t)M, K};
  for (int b = lane; b < nblk; b += 64) {
    uint4 q[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) q[j] = xr[4 * b + j];
    float y[32];
    unpack_bf16x32(q, y);
    const BlockOut d = block_out(o, row, b);
    block_mx<PAT>(y, d.spc, d.spm, d.sps, d.dnc, d.dns);
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers (called from the C ABI after validation)
// ---------------------------------------------------------------------------

template <int PAT>
static hipError_t launch_prep_mx_pat(const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* gamma, float eps,
                                     uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns,
                                     hipStream_t st) {
  dim3 grid((unsigned)((M + 3) / 4)), block(256);
  if (gamma == nullptr) {
    k_prep_mx_plain<PAT><<<grid, block, 0, st>>>(X, M, K, ldx, spc, spm, sps, dnc, dns);
  } else {
    const int chunks = (K / 32 + 63) / 64;
    if (chunks <= 1)
      k_prep_mx_norm<1, PAT><<<grid, block, 0, st>>>(X, M, K, ldx, gamma, eps, spc, spm, sps, dnc, dns);
    else if (chunks <= 2)
      k_prep_mx_norm<2, PAT><<<grid, block, 0, st>>>(X, M, K, ldx, gamma, eps, spc, spm, sps, dnc, dns);
    else if (chunks <= 4)
      k_prep_mx_norm<4, PAT><<<grid, block, 0, st>>>(X, M, K, ldx, gamma, eps, spc, spm, sps, dnc, dns);
    else
      k_prep_mx_norm<8, PAT><<<grid, block, 0, st>>>(X, M, K, ldx, gamma, eps, spc, spm, sps, dnc, dns);
  }
  return hipGetLastError();
}

hipError_t launch_prep_mx(const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* gamma, float eps, int pat,
                          uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns, hipStream_t st) {
  if (pat == 24) return launch_prep_mx_pat<24>(X, M, K, ldx, gamma, eps, spc, spm, sps, dnc, dns, st);
  return launch_prep_mx_pat<48>(X, M, K, ldx, gamma, eps, spc, spm, sps, dnc, dns, st);
}

}  // namespace sharq
