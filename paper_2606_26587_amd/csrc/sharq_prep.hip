// Fused SharQ activation preparation for gfx950 (SharQ Sec. 3.4, "Fused
// sparse-residual preparation"; Fig. 2).
//
// Every 32-element block is handled by one lane, so every block-local step
// (N:M selection inside groups of 4 or 8, the block max behind each scale, the
// residual) runs inside that lane without cross-lane traffic; only the RMSNorm
// sum of squares crosses lanes (and, for HiF4, a unit's maximum crosses a lane
// pair).  With RMSNorm a row is spread over 1, 2 or 4 wavefronts (or held as
// several blocks per lane for long rows); without it, one thread takes one
// block.  Every row is read from HBM once and every output byte is written
// once.
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


#include "sharq_prep_block.hpp"

#pragma clang fp contract(off)

namespace sharq {

// RMSNorm variant: the row's blocks stay in registers between the sum of
// squares and the quantization.  NB = blocks per lane, a power of two.
// NVFP4 reads the per-tensor scale S from S_ptr.
template <int NB, int PAT, bool NV, bool RES>
__global__ __launch_bounds__(256) void k_prep_norm(XSrc src, int M, int K, const uint16_t* __restrict__ gamma,
                                                   float eps, ActOut o, const float* S_ptr) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;   // whole wavefront; the kernel has no block barrier
  const int nblk = K / 32;
  const float S = NV ? *S_ptr : 1.0f, six_s = 6.0f * S;
  uint4 xs[NB][4];
  const float r = load_row_rms<NB, RES>(src, row, true, lane, nblk, K, eps, xs);
  if (o.dbg_r && lane == 0) o.dbg_r[row] = r;
  const uint4* gr = reinterpret_cast<const uint4*>(gamma);
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int b = lane + 64 * i;
    if (b >= nblk) break;
    uint4 gq[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) gq[j] = gr[4 * b + j];
    float y[32];
    norm_block(xs[i], gq, r, y);
    block_out_write<PAT, NV>(y, o, row, b, S, six_s);
  }
}

// RMSNorm variant with C wavefronts per row (C = 1, 2, 4; K <= 64 C blocks):
// wavefront c owns blocks 64 c + lane, so each lane holds one block.  Each
// wavefront reduces its 2048-position chunk with the in-lane tree and the
// lane butterfly; the C chunk sums meet in LDS and are added pairwise -- the
// same balanced tree as the one-wavefront-per-row kernel.  One group of 4 / C
// rows per workgroup: load, reduce, quantize, store, with no loop-carried
// state (a persistent form that prefetched the next group measured slower).
template <int C, int PAT, bool NV, bool RES>
__global__ __launch_bounds__(256) void k_prep_norm_split(XSrc src, int M, int K, const uint16_t* __restrict__ gamma,
                                                         float eps, ActOut o, const float* S_ptr) {
  __shared__ float part[4];
  constexpr int RPG = 4 / C;   // rows per workgroup
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int nblk = K / 32, b = (wave % C) * 64 + lane;
  const float S = NV ? *S_ptr : 1.0f, six_s = 6.0f * S;
  int64_t row = (int64_t)blockIdx.x * RPG + wave / C;
  const bool real = row < M;
  if (!real) row = M - 1;   // loads stay in bounds; only real rows store
  // lanes past the row's last block (K < 64 C blocks) read that block again
  // and add 0 to the sum; they store nothing
  const bool live = b < nblk;
  const int bl = live ? b : nblk - 1;
  uint4 gq[4], xq[4];
  // the gamma block is loaded with the row, before the reduction, so that its
  // latency is not on the path after it
  const uint4* gr = reinterpret_cast<const uint4*>(gamma);
#pragma unroll
  for (int j = 0; j < 4; ++j) gq[j] = gr[4 * bl + j];
  load_block<RES>(src, row, bl, xq, real && live);
  float x[32];
  unpack_bf16x32(xq, x);
  const float bs = block_sum_sq(x);
  const float cs = wave_tree_sum(live ? bs : 0.0f);
  float total = cs;
  if (C > 1) {
    if (lane == 0) part[wave] = cs;
    __syncthreads();
    const int base = (wave / C) * C;
    if (C == 2) total = part[base] + part[base + 1];
    else total = (part[base] + part[base + 1]) + (part[base + 2] + part[base + 3]);
  }
  const float r = (float)(1.0 / __builtin_sqrt((double)total / (double)K + (double)eps));
  if (o.dbg_r && real && lane == 0 && wave % C == 0) o.dbg_r[row] = r;
  if (real && live) {
    float y[32];
    norm_block(xq, gq, r, y);
    block_out_write<PAT, NV>(y, o, row, b, S, six_s);
  }
}

// Variant without RMSNorm: every block is independent, one thread per block.
// Grid (x, y) = (threads over one panel's blocks, panel): thread t of panel
// p takes block number V = 4 M p + t of the panel-major order, so
// consecutive threads write consecutive bytes of every output buffer (and
// read 256-byte row pieces of X).  The last panel may hold q < 4 blocks per
// row.
template <int PAT, bool NV, int SRC>
__global__ __launch_bounds__(256) void k_prep_blocks(XSrc src, int M, int K, ActOut o, const float* S_ptr) {
  const int nblk = K / 32, p = blockIdx.y;
  const int q = min(4, nblk - 4 * p);      // blocks per row in this panel
  const uint32_t t = blockIdx.x * 256u + threadIdx.x;
  if (t >= (uint32_t)q * (uint32_t)M) return;
  uint32_t row, j;
  if (q == 4) {
    row = t >> 2;
    j = t & 3u;
  } else {
    row = t / (uint32_t)q;
    j = t - row * (uint32_t)q;
  }
  const int b = 4 * p + (int)j;
  const float S = NV ? *S_ptr : 1.0f, six_s = 6.0f * S;
  uint4 xq[4];
  load_block<SRC>(src, (int64_t)row, b, xq, true);
  float y[32];
  unpack_bf16x32(xq, y);
  const BlockOut d = block_at<NV>(o, (int64_t)p * M * 4 + t);
  if (NV) {
    block_nv<PAT>(y, S, six_s, d);
  } else {
    block_mx<PAT>(y, d, o.rule_bias);
  }
}

// ---------------------------------------------------------------------------
// NVFP4 per-tensor scale (App. A.1.3): S = amax(y) / 2688 over the whole call,
// 1 for an all-zero tensor.  The running maximum is kept as the bit pattern
// of a non-negative float in the output's tensor_scale slot (bit patterns of
// non-negative floats order like the floats), then replaced by S.
// ---------------------------------------------------------------------------

__global__ void k_store_u32(uint32_t* p, uint32_t v) { *p = v; }

__global__ void k_copy_f32(const float* src, float* dst) { *dst = *src; }

__global__ void k_pts_finalize(uint32_t* slot) {
  const float amax = __uint_as_float(*slot);
  const float S = amax > 0.0f ? amax / 2688.0f : 1.0f;
  *reinterpret_cast<float*>(slot) = S;
}

// The pre-pass walks row groups grid-stride (one row per wavefront at a
// time) and issues one atomicMax per workgroup: atomics on one address
// serialize (~12 ns each measured), so one per row cost ~25 us at M = 2048.
// The grid is capped at kAmaxWG workgroups.
constexpr int kAmaxWG = 256;

__device__ __forceinline__ void amax_publish(float m, uint32_t* slot, float* wmax) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  m = wave_max(m);
  if (lane == 0) wmax[wave] = m;
  __syncthreads();
  if (threadIdx.x == 0) atomicMax(slot, __float_as_uint(fmaxf(fmaxf(wmax[0], wmax[1]), fmaxf(wmax[2], wmax[3]))));
}

template <int NB, bool RES>
__global__ __launch_bounds__(256) void k_amax_norm(XSrc src, int M, int K, const uint16_t* __restrict__ gamma,
                                                   float eps, uint32_t* slot) {
  __shared__ float wmax[4];
  const int lane = threadIdx.x & 63;
  const int nblk = K / 32;
  const uint4* gr = reinterpret_cast<const uint4*>(gamma);
  float m = 0.0f;
  for (int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); row < M; row += (int64_t)gridDim.x * 4) {
    uint4 xs[NB][4];
    const float r = load_row_rms<NB, RES>(src, row, false, lane, nblk, K, eps, xs);
#pragma unroll
    for (int i = 0; i < NB; ++i) {
      const int b = lane + 64 * i;
      if (b >= nblk) break;
      uint4 gq[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) gq[j] = gr[4 * b + j];
      float y[32];
      norm_block(xs[i], gq, r, y);
      m = fmaxf(m, absmax32(y));
    }
  }
  amax_publish(m, slot, wmax);   // every wavefront reaches the barrier inside
}

template <int SRC>
__global__ __launch_bounds__(256) void k_amax_plain(XSrc src, int M, int K, uint32_t* slot) {
  __shared__ float wmax[4];
  const int lane = threadIdx.x & 63;
  float m = 0.0f;
  for (int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6); row < M; row += (int64_t)gridDim.x * 4) {
    for (int b = lane; b < K / 32; b += 64) {
      uint4 q[4];
      load_block<SRC>(src, row, b, q, false);
      float y[32];
      unpack_bf16x32(q, y);
      m = fmaxf(m, absmax32(y));
    }
  }
  amax_publish(m, slot, wmax);
}

// ---------------------------------------------------------------------------
// Path combinations (Sec. 4.4, table "ablation-combination"; Sec. 3.1 eq.
// "direct-sparse-quant").  Path 1 quantizes y, path 2 the residual of y
// against path 1's dequantized values.  A sparse path keeps the top n of every
// m of its own input and quantizes the kept values per 32 logical positions
// (the backbone quantizer above); a dense path is the format's plain
// quantizer (MXFP4 per 32, NVFP4 per 16).  Path 1 is stored in the sp_*
// buffers and path 2 in the dn_* buffers (plus dn_meta for a sparse path 2),
// each with the block layout of its kind.
// ---------------------------------------------------------------------------

enum PathKind { kPathNone = 0, kPathSparse = 1, kPathDense = 2 };

// mode ids of the C interface: 1 sparse, 2 dense (RTN), 3 dense+dense,
// 4 sparse+sparse (0, the method itself, runs the kernels above)
__host__ __device__ constexpr int path1_kind(int mode) {
  return mode == 2 ? kPathNone : (mode == 3 ? kPathDense : kPathSparse);
}
__host__ __device__ constexpr int path2_kind(int mode) {
  return mode == 1 ? kPathNone : (mode == 4 ? kPathSparse : kPathDense);
}

struct PathBufs {
  uint8_t *c1, *m1, *s1, *c2, *m2, *s2;
  int64_t M;
  int K;
};

template <int PAT, class Q>
__device__ __forceinline__ void backbone_of(const float (&v)[32], const Q& qz, uint32_t (&codes)[2], uint32_t& meta,
                                            float (&R)[32]) {
  if (PAT == 24)
    backbone_24(v, qz, codes, meta, R);
  else if (PAT == 49)
    backbone_48p(v, qz, codes, meta, R);
  else
    backbone_48(v, qz, codes, meta, R);
}

// One path of kind KIND applied to the 32 values v of block number V (the
// panel-major block order of block_index): its codes / metadata / scales are
// stored, and R receives v minus the path's dequantized values.
template <int KIND, int PAT, bool NV>
__device__ __forceinline__ void path_block(const float (&v)[32], float S, float six_s, uint8_t* __restrict__ c,
                                           uint8_t* __restrict__ mt, uint8_t* __restrict__ sc, int64_t V,
                                           float (&R)[32]) {
  if (KIND == kPathSparse) {
    // the group maximum is always kept, so the kept values' block max is v's
    uint32_t codes[2], meta;
    if (NV) {
      const NvQ q = NvQ::make(absmax32(v), six_s, S);
      backbone_of<PAT>(v, q, codes, meta, R);
      sc[V] = (uint8_t)e4m3_bits(q.d);
    } else {
      const int e = mx_exponent(__float_as_uint(absmax32(v)));
      backbone_of<PAT>(v, MxQ::make(e), codes, meta, R);
      sc[V] = (uint8_t)(e + 127);
    }
    *reinterpret_cast<uint2*>(c + V * 8) = make_uint2(codes[0], codes[1]);
    *reinterpret_cast<uint32_t*>(mt + V * 4) = meta;
  } else {
    uint32_t w[4];
    if (NV) {
      const NvQ q0 = NvQ::make(absmax16(v), six_s, S), q1 = NvQ::make(absmax16(v + 16), six_s, S);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const NvQ& q = i < 2 ? q0 : q1;
        w[i] = enc8(v + 8 * i, q);
        const v2f d0 = q.template dec2<0>(w[i]), d1 = q.template dec2<1>(w[i]);
        const v2f d2 = q.template dec2<2>(w[i]), d3 = q.template dec2<3>(w[i]);
        R[8 * i + 0] = v[8 * i + 0] - d0.x; R[8 * i + 1] = v[8 * i + 1] - d0.y;
        R[8 * i + 2] = v[8 * i + 2] - d1.x; R[8 * i + 3] = v[8 * i + 3] - d1.y;
        R[8 * i + 4] = v[8 * i + 4] - d2.x; R[8 * i + 5] = v[8 * i + 5] - d2.y;
        R[8 * i + 6] = v[8 * i + 6] - d3.x; R[8 * i + 7] = v[8 * i + 7] - d3.y;
      }
      sc[V * 2] = (uint8_t)e4m3_bits(q0.d);
      sc[V * 2 + 1] = (uint8_t)e4m3_bits(q1.d);
    } else {
      const int e = mx_exponent(__float_as_uint(absmax32(v)));
      const MxQ q = MxQ::make(e);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        w[i] = enc8(v + 8 * i, q);
        const v2f d0 = q.template dec2<0>(w[i]), d1 = q.template dec2<1>(w[i]);
        const v2f d2 = q.template dec2<2>(w[i]), d3 = q.template dec2<3>(w[i]);
        R[8 * i + 0] = v[8 * i + 0] - d0.x; R[8 * i + 1] = v[8 * i + 1] - d0.y;
        R[8 * i + 2] = v[8 * i + 2] - d1.x; R[8 * i + 3] = v[8 * i + 3] - d1.y;
        R[8 * i + 4] = v[8 * i + 4] - d2.x; R[8 * i + 5] = v[8 * i + 5] - d2.y;
        R[8 * i + 6] = v[8 * i + 6] - d3.x; R[8 * i + 7] = v[8 * i + 7] - d3.y;
      }
      sc[V] = (uint8_t)(e + 127);
    }
    *reinterpret_cast<uint4*>(c + V * 16) = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

template <int MODE, int PAT, bool NV>
__device__ __forceinline__ void mode_block(const float (&y)[32], const PathBufs& o, int64_t V, float S, float six_s) {
  constexpr int K1 = path1_kind(MODE), K2 = path2_kind(MODE);
  float R[32];
  if (K1 != kPathNone) {
    path_block<K1, PAT, NV>(y, S, six_s, o.c1, o.m1, o.s1, V, R);
  } else {
#pragma unroll
    for (int k = 0; k < 32; ++k) R[k] = y[k];
  }
  if (K2 != kPathNone) {
    float R2[32];   // the second path's own residual is not used
    path_block<K2, PAT, NV>(R, S, six_s, o.c2, o.m2, o.s2, V, R2);
  }
}

// RMSNorm reciprocal of one row from a first pass over it (NB chunks of 2048
// positions, K <= 2048 NB): the balanced tree of the other kernels, with the
// chunks past the row adding exact zeros.
template <int NB>
__device__ __forceinline__ float row_rms_2pass(const XSrc& src, int64_t row, int lane, int nblk, int K, float eps) {
  float chunk[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int b = lane + 64 * i;
    float ss = 0.0f;
    if (b < nblk) {
      uint4 q[4];
      load_block<false>(src, row, b, q, false);
      float x[32];
      unpack_bf16x32(q, x);
      ss = block_sum_sq(x);
    }
    chunk[i] = wave_tree_sum(ss);
  }
#pragma unroll
  for (int w = NB / 2; w >= 1; w >>= 1)
#pragma unroll
    for (int k = 0; k < w; ++k) chunk[k] = chunk[2 * k] + chunk[2 * k + 1];
  return (float)(1.0 / __builtin_sqrt((double)chunk[0] / (double)K + (double)eps));
}

// One wavefront per row (4 rows per workgroup), lane l owning blocks
// l, l + 64, ...  With RMSNorm (NORM) the row is read twice: a first pass
// forms the same balanced tree as the other kernels (in-lane block sums, the
// lane butterfly per 2048-position chunk, the chunks pairwise; chunks past the
// row add exact zeros), a second pass quantizes.  Not a tuned kernel: the path
// combinations exist for ablation, not for the method's hot path.
template <int MODE, int PAT, bool NV, bool NORM>
__global__ __launch_bounds__(256) void k_prep_mode(XSrc src, int M, int K, const uint16_t* __restrict__ gamma,
                                                   float eps, PathBufs o, const float* S_ptr) {
  constexpr int NB = 8;   // chunks of 2048 positions (K <= 16384 with RMSNorm)
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;   // whole wavefront; the kernel has no block barrier
  const int nblk = K / 32;
  const float S = NV ? *S_ptr : 1.0f, six_s = 6.0f * S;
  const float r = NORM ? row_rms_2pass<NB>(src, row, lane, nblk, K, eps) : 1.0f;
  const uint4* gr = reinterpret_cast<const uint4*>(gamma);
  for (int b = lane; b < nblk; b += 64) {
    uint4 q[4];
    load_block<false>(src, row, b, q, false);
    float y[32];
    if (NORM) {
      uint4 gq[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) gq[j] = gr[4 * b + j];
      norm_block(q, gq, r, y);
    } else {
      unpack_bf16x32(q, y);
    }
    mode_block<MODE, PAT, NV>(y, o, block_index(o.M, o.K, row, b), S, six_s);
  }
}

// ---------------------------------------------------------------------------
// HiF4 preparation (2:4 backbone + dense residual).  A HiF4 unit of 64
// positions is the block pair (2u, 2u + 1), held by the lanes (2j, 2j + 1) of
// the row loop below; the unit maximum crosses the pair with one lane swap,
// everything else stays in the lane.  The backbone unit spans 64 logical
// positions: every group of 4 keeps its maximum, so its scales are those of
// the dense row.
// ---------------------------------------------------------------------------

struct HfScale {
  uint32_t code;   // E6M2
  float base, rec;
  uint32_t e8;     // this lane's 4 level-2 bits (bit i: values 8 i .. 8 i + 7 of its block)
  uint32_t e16;    // this lane's 8 level-3 bits (bit g: values 4 g .. 4 g + 3)
};

__device__ __forceinline__ HfScale hif4_scale(const float (&v)[32]) {
  float v16[8], v8[4];
#pragma unroll
  for (int g = 0; g < 8; ++g)
    v16[g] = fmaxf(fmaxf(fabsf(v[4 * g]), fabsf(v[4 * g + 1])), fmaxf(fabsf(v[4 * g + 2]), fabsf(v[4 * g + 3])));
#pragma unroll
  for (int i = 0; i < 4; ++i) v8[i] = fmaxf(v16[2 * i], v16[2 * i + 1]);
  const float bm = fmaxf(fmaxf(v8[0], v8[1]), fmaxf(v8[2], v8[3]));
  const float um = fmaxf(bm, __shfl_xor(bm, 1, 64));
  HfScale h;
  h.code = e6m2_code(um * kOneSeventhBf16);
  h.base = e6m2_value(h.code);
  h.rec = e6m2_rec(h.code);
  h.e8 = 0u;
  h.e16 = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) h.e8 |= (uint32_t)(v8[i] * h.rec >= 4.0f) << i;
#pragma unroll
  for (int g = 0; g < 8; ++g) h.e16 |= (uint32_t)(v16[g] * h.rec >= (((h.e8 >> (g >> 1)) & 1u) ? 4.0f : 2.0f)) << g;
  return h;
}

// micro-exponent of level-3 group g (0..7) of the lane's block
__device__ __forceinline__ int hif4_shift(const HfScale& h, int g) {
  return (int)(((h.e8 >> (g >> 1)) & 1u) + ((h.e16 >> g) & 1u));
}

// The unit's 4 metadata bytes [E6M2, E1_8, E1_16 low, E1_16 high] (valid in
// the even lane of the pair).
__device__ __forceinline__ uint32_t hif4_word(const HfScale& h) {
  const uint32_t mine = h.e8 | (h.e16 << 4);
  const uint32_t other = (uint32_t)__shfl_xor((int)mine, 1, 64);
  return h.code | (((mine & 0xFu) | ((other & 0xFu) << 4)) << 8) | (((mine >> 4) & 0xFFu) << 16) |
         (((other >> 4) & 0xFFu) << 24);
}

__device__ __forceinline__ uint32_t hif4_enc(float v, const HfScale& h, int sh) {
  return s1p2_code((v * h.rec) * exp2_int(-sh));
}

// 2:4 backbone of one block under HiF4: the selection and metadata of
// backbone_24, each kept value quantized with its level-3 group's scale.
__device__ __forceinline__ void backbone_24_hif4(const float (&y)[32], const HfScale& h, uint32_t (&codes)[2],
                                                 uint32_t& meta, float (&R)[32]) {
  codes[0] = codes[1] = 0u;
  meta = 0u;
#pragma unroll
  for (int g = 7; g >= 0; --g) {
    const float y0 = y[4 * g], y1 = y[4 * g + 1], y2 = y[4 * g + 2], y3 = y[4 * g + 3];
    lmask k0, k1, k2, k3;
    top2of4(y0, y1, y2, y3, k0, k1, k2, k3);
    const float v0 = lsel(k0, y0, lsel(k1, y1, y2));
    const float v1 = lsel(k3, y3, lsel(k2, y2, y1));
    meta = push_bit(meta, k3 | k2);
    meta = push_bit(meta, k3 | ~k2);
    meta = push_bit(meta, ~(k0 | k1));
    meta = push_bit(meta, k1 & ~k0);
    const int sh = hif4_shift(h, g);
    const uint32_t c0 = hif4_enc(v0, h, sh), c1 = hif4_enc(v1, h, sh);
    codes[g >> 2] |= (c0 | (c1 << 4)) << (8 * (g & 3));
    const float sc = h.base * exp2_int(sh);
    const float r0 = v0 - s1p2_value(c0, sc), r1 = v1 - s1p2_value(c1, sc);
    R[4 * g + 0] = lsel(k0, r0, y0);
    R[4 * g + 1] = lsel(k1, lsel(k0, r1, r0), y1);
    R[4 * g + 2] = lsel(k2, lsel(k3, r0, r1), y2);
    R[4 * g + 3] = lsel(k3, r1, y3);
  }
}

template <bool NORM>
__global__ __launch_bounds__(256) void k_prep_hif4(XSrc src, int M, int K, const uint16_t* __restrict__ gamma,
                                                   float eps, ActOut o) {
  const int lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= M) return;   // whole wavefront; the kernel has no block barrier
  const int nblk = K / 32;
  const float r = NORM ? row_rms_2pass<8>(src, row, lane, nblk, K, eps) : 1.0f;
  const uint4* gr = reinterpret_cast<const uint4*>(gamma);
  // nblk is even, so both lanes of a pair take the same iterations
  for (int b = lane; b < nblk; b += 64) {
    uint4 q[4];
    load_block<false>(src, row, b, q, false);
    float y[32];
    if (NORM) {
      uint4 gq[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) gq[j] = gr[4 * b + j];
      norm_block(q, gq, r, y);
    } else {
      unpack_bf16x32(q, y);
    }
    const HfScale hb = hif4_scale(y);
    uint32_t codes[2], meta;
    float R[32];
    backbone_24_hif4(y, hb, codes, meta, R);
    const HfScale hr = hif4_scale(R);
    uint32_t dn[4];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      uint32_t d = 0u;
#pragma unroll
      for (int i = 0; i < 8; ++i) d |= hif4_enc(R[8 * w + i], hr, hif4_shift(hr, 2 * w + (i >> 2))) << (4 * i);
      dn[w] = d;
    }
    const uint32_t wb = hif4_word(hb), wr = hif4_word(hr);
    const int64_t V = block_index(o.M, o.K, row, b);
    *reinterpret_cast<uint2*>(o.spc + V * 8) = make_uint2(codes[0], codes[1]);
    *reinterpret_cast<uint32_t*>(o.spm + V * 4) = meta;
    *reinterpret_cast<uint4*>(o.dnc + V * 16) = make_uint4(dn[0], dn[1], dn[2], dn[3]);
    if ((lane & 1) == 0) {   // the unit's metadata at the even block's 2-byte slots
      *reinterpret_cast<uint32_t*>(o.sps + V * 2) = wb;
      *reinterpret_cast<uint32_t*>(o.dns + V * 2) = wr;
    }
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers (called from the C ABI after validation)
// ---------------------------------------------------------------------------

template <int PAT, bool NV, bool RES>
static void go_prep(const XSrc& src, int M, int K, const uint16_t* gamma, float eps, const ActOut& o,
                    const float* S_ptr, dim3 grid, hipStream_t st) {
  dim3 block(256);
  const int nblk = K / 32;
  if (gamma == nullptr) {
    const dim3 g2((unsigned)((4 * (int64_t)M + 255) / 256), (unsigned)((nblk + 3) / 4));
    k_prep_blocks<PAT, NV, RES ? 1 : 0><<<g2, block, 0, st>>>(src, M, K, o, S_ptr);
    return;
  }
  if (nblk <= 256) {
    const int C = nblk <= 64 ? 1 : (nblk <= 128 ? 2 : 4);
    const dim3 g1((unsigned)((M + 4 / C - 1) / (4 / C)));
    if (C == 1) k_prep_norm_split<1, PAT, NV, RES><<<g1, block, 0, st>>>(src, M, K, gamma, eps, o, S_ptr);
    else if (C == 2) k_prep_norm_split<2, PAT, NV, RES><<<g1, block, 0, st>>>(src, M, K, gamma, eps, o, S_ptr);
    else k_prep_norm_split<4, PAT, NV, RES><<<g1, block, 0, st>>>(src, M, K, gamma, eps, o, S_ptr);
    return;
  }
  const int chunks = (K / 32 + 63) / 64;
  if (chunks <= 1)
    k_prep_norm<1, PAT, NV, RES><<<grid, block, 0, st>>>(src, M, K, gamma, eps, o, S_ptr);
  else if (chunks <= 2)
    k_prep_norm<2, PAT, NV, RES><<<grid, block, 0, st>>>(src, M, K, gamma, eps, o, S_ptr);
  else if (chunks <= 4)
    k_prep_norm<4, PAT, NV, RES><<<grid, block, 0, st>>>(src, M, K, gamma, eps, o, S_ptr);
  else
    k_prep_norm<8, PAT, NV, RES><<<grid, block, 0, st>>>(src, M, K, gamma, eps, o, S_ptr);
}

template <bool RES>
static void go_amax(const XSrc& src, int M, int K, const uint16_t* gamma, float eps, uint32_t* slot, dim3 rows_grid,
                    hipStream_t st) {
  const dim3 grid(rows_grid.x < (unsigned)kAmaxWG ? rows_grid.x : (unsigned)kAmaxWG);
  if (gamma == nullptr) {
    k_amax_plain<RES ? 1 : 0><<<grid, 256, 0, st>>>(src, M, K, slot);
    return;
  }
  const int chunks = (K / 32 + 63) / 64;
  if (chunks <= 1) k_amax_norm<1, RES><<<grid, 256, 0, st>>>(src, M, K, gamma, eps, slot);
  else if (chunks <= 2) k_amax_norm<2, RES><<<grid, 256, 0, st>>>(src, M, K, gamma, eps, slot);
  else if (chunks <= 4) k_amax_norm<4, RES><<<grid, 256, 0, st>>>(src, M, K, gamma, eps, slot);
  else k_amax_norm<8, RES><<<grid, 256, 0, st>>>(src, M, K, gamma, eps, slot);
}

template <bool RES>
static void go_prep_pat(int pat, bool nv, const XSrc& src, int M, int K, const uint16_t* gamma, float eps,
                        const ActOut& o, const float* S_ptr, dim3 grid, hipStream_t st) {
  if (nv) {
    if (pat == 24) go_prep<24, true, RES>(src, M, K, gamma, eps, o, S_ptr, grid, st);
    else if (pat == 49) go_prep<49, true, RES>(src, M, K, gamma, eps, o, S_ptr, grid, st);
    else go_prep<48, true, RES>(src, M, K, gamma, eps, o, S_ptr, grid, st);
  } else {
    if (pat == 24) go_prep<24, false, RES>(src, M, K, gamma, eps, o, nullptr, grid, st);
    else if (pat == 49) go_prep<49, false, RES>(src, M, K, gamma, eps, o, nullptr, grid, st);
    else go_prep<48, false, RES>(src, M, K, gamma, eps, o, nullptr, grid, st);
  }
}

// nv: NVFP4 with the per-tensor scale written to ts_out (from ts_in when
// given, else computed from the data).  res / h: the residual input and the
// h output of the fused residual add (both NULL without it).
hipError_t launch_prep(const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* res, int64_t ldr, uint16_t* h,
                       int64_t ldh, const uint16_t* gamma, float eps, int pat, bool nv, const float* ts_in,
                       float* ts_out, uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns,
                       uint8_t* spd, PrepExtras ex, hipStream_t st) {
  const ActOut o{spc, spm, sps, dnc, dns, (int64_t)M, K, spd, ex.rule_bias, ex.dbg_mask, ex.dbg_r};
  const XSrc src{X, ldx, res, ldr, h, ldh};
  const dim3 grid((unsigned)((M + 3) / 4));
  if (nv) {
    if (ts_in) {
      k_copy_f32<<<1, 1, 0, st>>>(ts_in, ts_out);
    } else {
      uint32_t* slot = reinterpret_cast<uint32_t*>(ts_out);
      k_store_u32<<<1, 1, 0, st>>>(slot, 0u);
      if (res) go_amax<true>(src, M, K, gamma, eps, slot, grid, st);
      else go_amax<false>(src, M, K, gamma, eps, slot, grid, st);
      k_pts_finalize<<<1, 1, 0, st>>>(slot);
    }
  }
  if (res) go_prep_pat<true>(pat, nv, src, M, K, gamma, eps, o, ts_out, grid, st);
  else go_prep_pat<false>(pat, nv, src, M, K, gamma, eps, o, ts_out, grid, st);
  return hipGetLastError();
}

template <int MODE, int PAT, bool NV>
static void go_prep_mode(const XSrc& src, int M, int K, const uint16_t* gamma, float eps, const PathBufs& o,
                         const float* S_ptr, dim3 grid, hipStream_t st) {
  if (gamma)
    k_prep_mode<MODE, PAT, NV, true><<<grid, 256, 0, st>>>(src, M, K, gamma, eps, o, S_ptr);
  else
    k_prep_mode<MODE, PAT, NV, false><<<grid, 256, 0, st>>>(src, M, K, gamma, eps, o, S_ptr);
}

template <int MODE, bool NV>
static void go_prep_mode_pat(int pat, const XSrc& src, int M, int K, const uint16_t* gamma, float eps,
                             const PathBufs& o, const float* S_ptr, dim3 grid, hipStream_t st) {
  if (path1_kind(MODE) != kPathSparse && path2_kind(MODE) != kPathSparse)
    go_prep_mode<MODE, 24, NV>(src, M, K, gamma, eps, o, S_ptr, grid, st);   // the pattern is not used
  else if (pat == 24)
    go_prep_mode<MODE, 24, NV>(src, M, K, gamma, eps, o, S_ptr, grid, st);
  else if (pat == 49)
    go_prep_mode<MODE, 49, NV>(src, M, K, gamma, eps, o, S_ptr, grid, st);
  else
    go_prep_mode<MODE, 48, NV>(src, M, K, gamma, eps, o, S_ptr, grid, st);
}

// Preparation of a path combination (mode 1-4; see PathKind).  Buffers c1,
// m1, s1 receive path 1 and c2, m2, s2 path 2, in the layout of their kinds.
hipError_t launch_prep_mode(int mode, const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* gamma, float eps,
                            int pat, bool nv, const float* ts_in, float* ts_out, uint8_t* c1, uint8_t* m1,
                            uint8_t* s1, uint8_t* c2, uint8_t* m2, uint8_t* s2, hipStream_t st) {
  const PathBufs o{c1, m1, s1, c2, m2, s2, (int64_t)M, K};
  const XSrc src{X, ldx, nullptr, 0, nullptr, 0};
  const dim3 grid((unsigned)((M + 3) / 4));
  if (nv) {
    if (ts_in) {
      k_copy_f32<<<1, 1, 0, st>>>(ts_in, ts_out);
    } else {
      uint32_t* slot = reinterpret_cast<uint32_t*>(ts_out);
      k_store_u32<<<1, 1, 0, st>>>(slot, 0u);
      go_amax<false>(src, M, K, gamma, eps, slot, grid, st);
      k_pts_finalize<<<1, 1, 0, st>>>(slot);
    }
  }
  const float* S = nv ? ts_out : nullptr;
  switch (mode) {
    case 1: nv ? go_prep_mode_pat<1, true>(pat, src, M, K, gamma, eps, o, S, grid, st)
               : go_prep_mode_pat<1, false>(pat, src, M, K, gamma, eps, o, S, grid, st); break;
    case 2: nv ? go_prep_mode_pat<2, true>(pat, src, M, K, gamma, eps, o, S, grid, st)
               : go_prep_mode_pat<2, false>(pat, src, M, K, gamma, eps, o, S, grid, st); break;
    case 3: nv ? go_prep_mode_pat<3, true>(pat, src, M, K, gamma, eps, o, S, grid, st)
               : go_prep_mode_pat<3, false>(pat, src, M, K, gamma, eps, o, S, grid, st); break;
    case 4: nv ? go_prep_mode_pat<4, true>(pat, src, M, K, gamma, eps, o, S, grid, st)
               : go_prep_mode_pat<4, false>(pat, src, M, K, gamma, eps, o, S, grid, st); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// HiF4 preparation (2:4 backbone, SharQ mode; K a multiple of 64, K <= 16384
// with RMSNorm).
hipError_t launch_prep_hif4(const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* gamma, float eps,
                            uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns, hipStream_t st) {
  const ActOut o{spc, spm, sps, dnc, dns, (int64_t)M, K, nullptr, kE8Floor, nullptr, nullptr};
  const XSrc src{X, ldx, nullptr, 0, nullptr, 0};
  const dim3 grid((unsigned)((M + 3) / 4));
  if (gamma)
    k_prep_hif4<true><<<grid, 256, 0, st>>>(src, M, K, gamma, eps, o);
  else
    k_prep_hif4<false><<<grid, 256, 0, st>>>(src, M, K, gamma, eps, o);
  return hipGetLastError();
}

// Preparation of the down projection's input with SiLU.mul fused in front:
// h = bf16(SiLU(gate) * up), written to h (when not NULL) and prepared
// without RMSNorm.  nv: NVFP4 with the per-tensor scale from ts_in or from
// an amax pre-pass over h.
hipError_t launch_prep_silu(const uint16_t* gate, const uint16_t* up, uint16_t* h, int M, int K, int64_t ldg,
                            int64_t ldu, int64_t ldh, int pat, bool nv, const float* ts_in, float* ts_out,
                            uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns, uint8_t* spd,
                            PrepExtras ex, hipStream_t st) {
  const ActOut o{spc, spm, sps, dnc, dns, (int64_t)M, K, spd, ex.rule_bias, ex.dbg_mask, nullptr};
  const XSrc src{gate, ldg, up, ldu, h, ldh};
  const dim3 grid((unsigned)((M + 3) / 4));
  if (nv) {
    if (ts_in) {
      k_copy_f32<<<1, 1, 0, st>>>(ts_in, ts_out);
    } else {
      uint32_t* slot = reinterpret_cast<uint32_t*>(ts_out);
      k_store_u32<<<1, 1, 0, st>>>(slot, 0u);
      k_amax_plain<2><<<grid, 256, 0, st>>>(src, M, K, slot);
      k_pts_finalize<<<1, 1, 0, st>>>(slot);
    }
  }
  const int nblk = K / 32;
  const dim3 g2((unsigned)((4 * (int64_t)M + 255) / 256), (unsigned)((nblk + 3) / 4));
  const float* S = nv ? ts_out : nullptr;
  if (nv) {
    if (pat == 24) k_prep_blocks<24, true, 2><<<g2, 256, 0, st>>>(src, M, K, o, S);
    else if (pat == 49) k_prep_blocks<49, true, 2><<<g2, 256, 0, st>>>(src, M, K, o, S);
    else k_prep_blocks<48, true, 2><<<g2, 256, 0, st>>>(src, M, K, o, S);
  } else {
    if (pat == 24) k_prep_blocks<24, false, 2><<<g2, 256, 0, st>>>(src, M, K, o, S);
    else if (pat == 49) k_prep_blocks<49, false, 2><<<g2, 256, 0, st>>>(src, M, K, o, S);
    else k_prep_blocks<48, false, 2><<<g2, 256, 0, st>>>(src, M, K, o, S);
  }
  return hipGetLastError();
}

}  // namespace sharq
