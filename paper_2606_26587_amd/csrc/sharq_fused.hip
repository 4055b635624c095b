// Small-M SharQ linear with the activation preparation in the GEMM's
// prologue (decode): one kernel instead of a preparation launch followed by
// a GEMM launch -- the "near-single-kernel data flow" of Sec. 4.3, with the
// fused preparation of Sec. 3.4 and the two-path output of Sec. 3.3 eq.
// "sharq-output".
//
// Every workgroup owns 16 NB output columns of all M (<= 16) rows, as in the
// small-M kernel.  It first prepares the M activation rows itself, into LDS:
// RMSNorm (the balanced-tree sum of squares, per-block sums then a tree over
// the blocks), the N:M mask, the backbone as dense codes and the residual,
// with their E8M0 scales -- the same block code as the preparation kernels,
// so the bytes are identical.  Workgroup 0 also writes the prepared
// activation to the caller's buffers.  The weight stream of the first two
// panels is issued before the preparation, so its latency overlaps it.  Then
// its KS wavefronts split K and run the 16x16x128 block-scaled FP4 MFMA over
// the LDS activation and the weight streamed from HBM, and the KS partial
// tiles are added in LDS in a fixed order.
//
// The preparation is repeated by every workgroup, so its cost grows with M
// while the separate preparation kernel's does not; the launcher uses this
// kernel for the few rows where that still wins.

#include "sharq_prep_block.hpp"

#pragma clang fp contract(off)

namespace sharq {

typedef float v4f_fused __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v8i as_operand_f(uint4 q) {
  v8i v;
  v[0] = (int)q.x; v[1] = (int)q.y; v[2] = (int)q.z; v[3] = (int)q.w;
  v[4] = 0; v[5] = 0; v[6] = 0; v[7] = 0;
  return v;
}

template <typename OutT>
__device__ __forceinline__ void fused_store(OutT* p, float v);
template <>
__device__ __forceinline__ void fused_store<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void fused_store<uint16_t>(uint16_t* p, float v) { *p = f32_to_bf16_rne(v); }
template <>
__device__ __forceinline__ void fused_store<_Float16>(_Float16* p, float v) { *p = (_Float16)v; }

// LDS layout of the prepared rows (M rows, nblk blocks of 32 positions):
// residual codes and dense backbone codes, 16 bytes per block each, then the
// backbone and residual E8M0 bytes, then the per-block sums of squares and
// the rows' r.
struct FusedLds {
  uint8_t *dn, *spd, *sps, *dns;
  float *bss, *r;
  int nblk;
};

__device__ __forceinline__ FusedLds fused_lds(uint8_t* base, int M, int nblk) {
  FusedLds l;
  const int nb = M * nblk;
  l.dn = base;
  l.spd = base + nb * 16;
  l.sps = base + nb * 32;
  l.dns = base + nb * 33;
  l.bss = reinterpret_cast<float*>(base + ((nb * 34 + 15) & ~15));
  l.r = l.bss + nb;
  l.nblk = nblk;
  return l;
}

// LDS bytes of the prepared rows and their reduction scratch.
__host__ __device__ constexpr int fused_prep_lds_bytes(int M, int nblk) {
  return ((M * nblk * 34 + 15) & ~15) + 4 * M * nblk + 4 * 16;
}

template <int NB>
struct FusedWStage {
  uint4 w[NB];
  uint32_t ws[NB];
};

template <int NB>
__device__ __forceinline__ void fused_load_w(FusedWStage<NB>& st, const uint8_t* wc, const uint8_t* ws, int N, int n0,
                                             int ks, int lane) {
  const int j = lane >> 4;
  const int64_t pn = (int64_t)ks * N;
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    const int col = min(n0 + 16 * n + (lane & 15), N - 1);
    st.w[n] = *reinterpret_cast<const uint4*>(wc + (pn + col) * 64 + 16 * j);
    st.ws[n] = ws[(pn + col) * 4 + j];
  }
}

template <int NB, int KS, int PAT, typename OutT>
__global__ __launch_bounds__(64 * KS) void k_linear_mx_skinny_prep(XSrc src, int M, int K,
                                                                   const uint16_t* __restrict__ gamma, float eps,
                                                                   ActOut act, const uint8_t* wc, const uint8_t* ws,
                                                                   int N, OutT* Y, int64_t ldy) {
  extern __shared__ __attribute__((aligned(16))) uint8_t fused_smem[];
  constexpr int T = 64 * KS;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int nblk = K / 32, nks = K / 128;
  const FusedLds L = fused_lds(fused_smem, M, nblk);
  float* part = reinterpret_cast<float*>(fused_smem + fused_prep_lds_bytes(M, nblk));   // [KS-1][NB][64][4]
  const int n0 = blockIdx.x * 16 * NB;
  const int per = (nks + KS - 1) / KS;
  const int k0 = wave * per, k1 = min(nks, k0 + per);

  // the first two weight panels go out before the preparation
  FusedWStage<NB> s0, s1;
  if (k0 < k1) fused_load_w<NB>(s0, wc, ws, N, n0, k0, lane);
  if (k0 + 1 < k1) fused_load_w<NB>(s1, wc, ws, N, n0, k0 + 1, lane);

  // ---- preparation of the M rows into LDS (workgroup 0: also to `act`)
  const int pairs = M * nblk;
  if (gamma != nullptr) {
    for (int i = tid; i < pairs; i += T) {
      uint4 q[4];
      load_block<0>(src, i / nblk, i % nblk, q, false);
      float x[32];
      unpack_bf16x32(q, x);
      L.bss[i] = block_sum_sq(x);
    }
    __syncthreads();
    // per row: the balanced tree over its blocks (padded with zeros to a
    // power of two of at least 64 blocks, which adds exact zeros): lane l
    // sums its aligned run of c blocks pairwise, then the xor butterfly
    int P = 64;
    while (P < nblk) P *= 2;
    const int c = P / 64;
    for (int row = wave; row < M; row += KS) {
      float s[8];
      for (int u = 0; u < c; ++u) {
        const int b = lane * c + u;
        s[u] = b < nblk ? L.bss[row * nblk + b] : 0.0f;
      }
      for (int w = c / 2; w >= 1; w >>= 1)
        for (int u = 0; u < w; ++u) s[u] = s[2 * u] + s[2 * u + 1];
      const float total = wave_tree_sum(s[0]);
      if (lane == 0) L.r[row] = (float)(1.0 / __builtin_sqrt((double)total / (double)K + (double)eps));
    }
    __syncthreads();
  }
  for (int i = tid; i < pairs; i += T) {
    const int row = i / nblk, b = i % nblk;
    uint4 q[4];
    load_block<0>(src, row, b, q, false);
    float y[32];
    if (gamma != nullptr) {
      uint4 gq[4];
      const uint4* gr = reinterpret_cast<const uint4*>(gamma);
#pragma unroll
      for (int j = 0; j < 4; ++j) gq[j] = gr[4 * b + j];
      norm_block(q, gq, L.r[row], y);
    } else {
      unpack_bf16x32(q, y);
    }
    BlockOut d;
    d.spc = nullptr;
    d.spm = nullptr;
    d.sps = L.sps + i;
    d.dnc = L.dn + 16 * i;
    d.dns = L.dns + i;
    d.spd = L.spd + 16 * i;
    d.dbg_mask = nullptr;
    block_mx<PAT>(y, d, act.rule_bias);
    if (blockIdx.x == 0) {
      block_out_write<PAT, false>(y, act, row, b, 1.0f, 6.0f);
      if (act.dbg_r != nullptr && gamma != nullptr && b == 0) act.dbg_r[row] = L.r[row];
    }
  }
  __syncthreads();

  // ---- two-path GEMM over the LDS activation
  v4f_fused acc[NB];
#pragma unroll
  for (int n = 0; n < NB; ++n) acc[n] = v4f_fused{0.0f, 0.0f, 0.0f, 0.0f};
  const int arow = min(lane & 15, M - 1);   // rows past M read row M - 1; their outputs are not stored
  const int j = lane >> 4;
  auto step = [&](const FusedWStage<NB>& st, int ks) {
    const int i = arow * nblk + 4 * ks + j;
    const v8i asp = as_operand_f(*reinterpret_cast<const uint4*>(L.spd + 16 * i));
    const v8i adn = as_operand_f(*reinterpret_cast<const uint4*>(L.dn + 16 * i));
    const int ssp = L.sps[i], sdn = L.dns[i];
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const v8i bw = as_operand_f(st.w[n]);
      acc[n] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(bw, asp, acc[n], 4, 4, 0, (int)st.ws[n], 0, ssp);
      acc[n] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(bw, adn, acc[n], 4, 4, 0, (int)st.ws[n], 0, sdn);
    }
  };
  int ks = k0;
  for (; ks + 1 < k1; ks += 2) {
    step(s0, ks);
    if (ks + 2 < k1) fused_load_w<NB>(s0, wc, ws, N, n0, ks + 2, lane);
    step(s1, ks + 1);
    if (ks + 3 < k1) fused_load_w<NB>(s1, wc, ws, N, n0, ks + 3, lane);
  }
  if (ks < k1) step(s0, ks);

  // partial tiles of wavefronts 1..KS-1 to LDS; wavefront 0 adds them in order
  if (wave > 0) {
#pragma unroll
    for (int n = 0; n < NB; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) part[(((wave - 1) * NB + n) * 64 + lane) * 4 + r] = acc[n][r];
  }
  __syncthreads();
  if (wave != 0) return;
  for (int w = 0; w < KS - 1; ++w)
#pragma unroll
    for (int n = 0; n < NB; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) acc[n][r] += part[((w * NB + n) * 64 + lane) * 4 + r];
  const int row = lane & 15;
  if (row >= M) return;
#pragma unroll
  for (int n = 0; n < NB; ++n)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int col = n0 + 16 * n + 4 * (lane >> 4) + r;
      if (col < N) fused_store<OutT>(Y + (int64_t)row * ldy + col, acc[n][r]);
    }
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------

// Rows up to which the fused kernel replaces the preparation launch + small-M
// GEMM launch (every workgroup repeats the preparation of all M rows).
constexpr int kFusedMaxM = 4;
constexpr int kFusedMaxLds = 64 * 1024;

// Column fragments and K split of the small-M GEMM at M <= 16, the same rule
// as the separate small-M kernel's (so the two give bit-identical outputs):
// 4 (2) fragments when N leaves at least 192 workgroups of 64 (32) columns,
// and a K split keeping about 8192 weight streams in flight with at least 4
// panels per wavefront (at most 8 wavefronts with 4 fragments).
static void fused_config(int N, int K, int& nb, int& ks) {
  nb = (N + 63) / 64 >= 192 ? 4 : (N + 31) / 32 >= 192 ? 2 : 1;
  const int cap = nb == 4 ? 8 : 16, wgs = (N + 15) / 16, nks = K / 128;
  ks = 4;
  while (ks < cap && wgs * ks * 2 <= 8192 && nks >= 4 * ks * 2) ks *= 2;
}

static size_t fused_lds_total(int M, int K, int nb, int ks) {
  return (size_t)fused_prep_lds_bytes(M, K / 32) + (size_t)(ks - 1) * nb * 64 * 16;
}

bool fused_prep_linear_applies(int64_t M, int K, int N) {
  if (M < 1 || M > kFusedMaxM || K % 128 != 0 || K > 16384 || N < 1) return false;
  int nb, ks;
  fused_config(N, K, nb, ks);
  return fused_lds_total((int)M, K, nb, ks) <= (size_t)kFusedMaxLds;
}

template <int NB, int KS, int PAT, typename OutT>
static hipError_t go_fused(const XSrc& src, int M, int K, const uint16_t* gamma, float eps, const ActOut& act,
                           const uint8_t* wc, const uint8_t* ws, int N, void* Y, int64_t ldy, hipStream_t st) {
  const int ncg = (N + 16 * NB - 1) / (16 * NB);
  const size_t lds = fused_lds_total(M, K, NB, KS);
  k_linear_mx_skinny_prep<NB, KS, PAT, OutT><<<dim3((unsigned)ncg), dim3(64 * KS), lds, st>>>(
      src, M, K, gamma, eps, act, wc, ws, N, reinterpret_cast<OutT*>(Y), ldy);
  return hipGetLastError();
}

template <int PAT, typename OutT>
static hipError_t go_fused_cfg(const XSrc& src, int M, int K, const uint16_t* gamma, float eps, const ActOut& act,
                               const uint8_t* wc, const uint8_t* ws, int N, void* Y, int64_t ldy, hipStream_t st) {
  int nb, ks;
  fused_config(N, K, nb, ks);
#define SHARQ_FUSED(NB_, KS_) \
  if (nb == NB_ && ks == KS_) return go_fused<NB_, KS_, PAT, OutT>(src, M, K, gamma, eps, act, wc, ws, N, Y, ldy, st);
  SHARQ_FUSED(4, 4) SHARQ_FUSED(4, 8)
  SHARQ_FUSED(2, 4) SHARQ_FUSED(2, 8) SHARQ_FUSED(2, 16)
  SHARQ_FUSED(1, 4) SHARQ_FUSED(1, 8) SHARQ_FUSED(1, 16)
#undef SHARQ_FUSED
  return hipErrorInvalidValue;   // unreachable: (nb, ks) is one of the above
}

// The preparation of X [M][K] into `act` and the two-path GEMM with the
// weight into Y, as one kernel (callers check fused_prep_linear_applies).
hipError_t launch_prep_linear_fused(const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* gamma, float eps,
                                    int pat, uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns,
                                    uint8_t* spd, PrepExtras ex, const uint8_t* wc, const uint8_t* ws, int N, int ydt,
                                    void* Y, int64_t ldy, hipStream_t st) {
  const ActOut act{spc, spm, sps, dnc, dns, (int64_t)M, K, spd, ex.rule_bias, ex.dbg_mask, ex.dbg_r};
  const XSrc src{X, ldx, nullptr, 0, nullptr, 0};
#define SHARQ_FUSED_DT(PAT_)                                                                                    \
  if (pat == PAT_) {                                                                                            \
    if (ydt == 2) return go_fused_cfg<PAT_, float>(src, M, K, gamma, eps, act, wc, ws, N, Y, ldy, st);          \
    if (ydt == 1) return go_fused_cfg<PAT_, _Float16>(src, M, K, gamma, eps, act, wc, ws, N, Y, ldy, st);       \
    return go_fused_cfg<PAT_, uint16_t>(src, M, K, gamma, eps, act, wc, ws, N, Y, ldy, st);                     \
  }
  SHARQ_FUSED_DT(24) SHARQ_FUSED_DT(48) SHARQ_FUSED_DT(49)
#undef SHARQ_FUSED_DT
  return hipErrorInvalidValue;
}

}  // namespace sharq
