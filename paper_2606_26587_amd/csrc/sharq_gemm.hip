// SharQ two-path FP4 GEMM for gfx950 (SharQ Sec. 3.3 eq. "sharq-output";
// Sec. 3.4 "Shared FP4 weights with path-specific scales" and "Residual path
// compensation by accumulation").
//
//   Y = dequant(backbone) * dequant(W)^T + dequant(residual) * dequant(W)^T
//
// Both products run on the CDNA4 block-scaled MFMA
// v_mfma_scale_f32_32x32x64_f8f6f4 with E2M1 operands and E8M0 scales, into
// ONE fp32 accumulator; Y is written once.
//
// gfx950 has no sparse MFMA for FP4 operands (the sparse smfmac forms take
// 8/16-bit inputs only), so the 2:4 or 4:8 backbone enters the MFMA as dense
// E2M1 nibbles with zeros at the dropped positions: either expanded from its
// compressed form in the registers of the wavefront that owns the rows (each
// wavefront owns 32 distinct rows of the 128-row tile, so a row is expanded
// once per tile and never goes through LDS), or read from the dense copy the
// preparation wrote (pattern 0), which spares every column tile the
// expansion.  The shared weight tile (E2M1 payload + E8M0 scales) is staged
// through LDS once per K step and read by both MFMAs of every fragment.
// Also here: the small-M kernel for decode, the grouped (MoE) form, the
// NVFP4 and HiF4 kernels on 16-bit MFMA over exactly dequantized operands
// (fp16 in the NVFP4 kernel for K a multiple of 128, bf16 elsewhere), and
// the generic kernels of the ablation path combinations.

// MFMA 32x32x64 FP4 operand layout (lane l, 64-wide wavefront): lane l holds
// row (l % 32) and the 32 K values of block (l / 32) of the 64-wide K slice as
// 32 nibbles in its first four dwords (lower K in the lower nibble); its
// 32-bit scale operand supplies, through op_sel, the E8M0 byte of that row and
// block.  Accumulator element r of lane l is output row
// 8 (r / 4) + 4 (l / 32) + (r % 4), column l % 32.

#include "sharq_device.hpp"
#include <type_traits>

namespace sharq {

constexpr int kBM = 128;          // tile rows: 4 wavefronts x 32
constexpr int kBK = 128;          // K per step: 4 scale blocks, 64 bytes of codes per row
constexpr int kLdsStride = 80;    // bytes per staged weight row (64 + 16 to spread LDS banks)
constexpr int kSkinnyMaxM = 32;   // activation rows up to which the small-M kernel runs
constexpr int kSkinnyMaxRowTiled = 256;   // ... and, when the main kernel has few tiles, up to this many

__device__ __forceinline__ v8i as_operand(uint4 q) {
  v8i v;
  v[0] = (int)q.x; v[1] = (int)q.y; v[2] = (int)q.z; v[3] = (int)q.w;
  v[4] = 0; v[5] = 0; v[6] = 0; v[7] = 0;
  return v;
}

// ---------------------------------------------------------------------------
// Per-lane activation fragment of one K step (two 64-wide MFMA sub-steps)
// ---------------------------------------------------------------------------

struct AStep {
  uint4 dn[2];       // residual codes, sub-step 0 / 1
  uint2 spc[2];      // compressed backbone codes
  uint32_t spm[2];   // backbone metadata
  uint32_t sdn, ssp; // E8M0 scales of the step's 4 blocks (byte j = block 4 ks + j)
  uint4 spd[2];      // the dense backbone codes instead (pattern 0: a dense copy was prepared)
};

// Activation rows live in panel-major buffers: K is cut into panels of 128
// positions (one K step; the last panel may be narrower) and panel p stores
// all R rows' bytes for its K range back to back, so the 32 rows of a
// wavefront are 2 KB (codes), 1 KB (backbone), 512 B (metadata) and 128 B
// (scales) of contiguous memory per step.
struct ARow {
  const uint8_t *dn, *spc, *spm, *dns, *sps;   // buffer bases
  int64_t r, R;                                // this lane's activation row, rows in the buffers
};

template <bool SCALE_DW>
__device__ __forceinline__ void load_a(AStep& s, const ARow& a, int ks, int half, int nblk, int K) {
  // SCALE_DW: K is a multiple of 128, every panel is full and every block exists
  const int wp = SCALE_DW ? 128 : min(128, K - 128 * ks);
  const int64_t pr = (int64_t)ks * a.R;
  const uint8_t* dn = a.dn + pr * 64 + a.r * (wp / 2);
  const uint8_t* spc = a.spc + pr * 32 + a.r * (wp / 4);
  const uint8_t* spm = a.spm + pr * 16 + a.r * (wp / 8);
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const int j = 2 * sub + half;   // block within the panel
    if (SCALE_DW || 4 * ks + j < nblk) {
      s.dn[sub] = *reinterpret_cast<const uint4*>(dn + 16 * j);
      s.spc[sub] = *reinterpret_cast<const uint2*>(spc + 8 * j);
      s.spm[sub] = *reinterpret_cast<const uint32_t*>(spm + 4 * j);
    } else {
      s.dn[sub] = make_uint4(0u, 0u, 0u, 0u);
      s.spc[sub] = make_uint2(0u, 0u);
      s.spm[sub] = 0x44444444u;   // 2:4: a valid (0,1) pair; 4:8 ignores it with zero codes
    }
  }
  const uint8_t* dns = a.dns + pr * 4 + a.r * (wp / 32);
  const uint8_t* sps = a.sps + pr * 4 + a.r * (wp / 32);
  if (SCALE_DW) {
    // raw dwords: the per-lane byte shift is applied at the point of use so
    // that no instruction waits on these loads before the MFMAs need them
    s.sdn = *reinterpret_cast<const uint32_t*>(dns);
    s.ssp = *reinterpret_cast<const uint32_t*>(sps);
  } else {
    // same byte order as the dword form: byte j = block 4 ks + j (127 past K)
    s.sdn = 0u;
    s.ssp = 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const bool ok = 4 * ks + j < nblk;
      s.sdn |= (uint32_t)(ok ? dns[j] : 127u) << (8 * j);
      s.ssp |= (uint32_t)(ok ? sps[j] : 127u) << (8 * j);
    }
  }
}

// The weight tile of one K step held in registers between its global load and
// its LDS store: BN rows x 64 bytes of codes (16 bytes per thread and chunk)
// plus one dword of four E8M0 scales per row.
template <int NF>
struct WStep {
  uint4 q[NF / 2];
  uint32_t s;
};

template <int NF, bool SCALE_DW>
__device__ __forceinline__ void load_w(WStep<NF>& w, const uint8_t* wc, const uint8_t* ws, int n0, int N, int K,
                                       int ks, int nblk) {
  // panel-major weight: panel ks holds all N rows' 64 bytes (or fewer for a
  // narrow last panel), so a full tile of BN rows is one contiguous run
  constexpr int BN = 32 * NF;
  const int tid = threadIdx.x;
  const int wp = SCALE_DW ? 128 : min(128, K - 128 * ks);
  const int64_t pn = (int64_t)ks * N;
#pragma unroll
  for (int j = 0; j < BN / 64; ++j) {
    const int c = tid + 256 * j;
    const int row = c >> 2, part = c & 3;
    const int n = min(n0 + row, N - 1);
    w.q[j] = (SCALE_DW || 4 * ks + part < nblk)
                 ? *reinterpret_cast<const uint4*>(wc + pn * 64 + (int64_t)n * (wp / 2) + 16 * part)
                 : make_uint4(0u, 0u, 0u, 0u);
  }
  // one scale dword per weight row (threads 0 .. BN-1).  Threads past BN
  // reread row BN-1 and never store it: no branch, which keeps the
  // interleaved K step one basic block (the compiler would otherwise move its
  // MFMAs out of their slots), and no select on the loaded value, which
  // would make the thread wait for the load where it is issued
  const int n = min(n0 + (BN >= 256 ? tid : min(tid, BN - 1)), N - 1);
  const uint8_t* sr = ws + pn * 4 + (int64_t)n * (wp / 32);
  uint32_t sv = 0u;
  if (SCALE_DW) {
    sv = *reinterpret_cast<const uint32_t*>(sr);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) sv |= (uint32_t)(4 * ks + j < nblk ? sr[j] : 127u) << (8 * j);
  }
  w.s = sv;
}

// Weight scales in LDS are laid out per (column, lane half): lane (col, h)
// finds, at byte 2f + sub of its 2 NF-byte record, the E8M0 scale of weight row
// f*32 + col for block 4 ks + 2 sub + h -- exactly the byte its MFMA for
// fragment f, sub-step sub needs -- so one LDS read fetches all of them and
// op_sel selects the byte.
template <int NF>
__device__ __forceinline__ void store_w(const WStep<NF>& w, uint8_t* lds_w, uint8_t* lds_s) {
  constexpr int BN = 32 * NF;
  const int tid = threadIdx.x;
#pragma unroll
  for (int j = 0; j < BN / 64; ++j) {
    const int c = tid + 256 * j;
    const int row = c >> 2, part = c & 3;
    *reinterpret_cast<uint4*>(lds_w + row * kLdsStride + 16 * part) = w.q[j];
  }
  if (BN >= 256 || tid < BN) {
    const int f = tid >> 5, col = tid & 31;
    // blocks 0 and 2 of the step go to half 0, blocks 1 and 3 to half 1
    const uint32_t h0 = __builtin_amdgcn_perm(0u, w.s, 0x0c0c0200u);   // b0 | b2 << 8
    const uint32_t h1 = __builtin_amdgcn_perm(0u, w.s, 0x0c0c0301u);   // b1 | b3 << 8
    *reinterpret_cast<uint16_t*>(lds_s + (2 * col + 0) * (2 * NF) + 2 * f) = (uint16_t)h0;
    *reinterpret_cast<uint16_t*>(lds_s + (2 * col + 1) * (2 * NF) + 2 * f) = (uint16_t)h1;
  }
}

template <int SA, int SB>
__device__ __forceinline__ v16f mfma_fp4(v8i a, v8i b, v16f c, uint32_t sa, uint32_t sb) {
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 4, 4, SA, (int)sa, SB, (int)sb);
}

template <int SUB, int NF>
__device__ __forceinline__ void mma_sub(v16f (&acc)[NF], const uint8_t* lds_w, const uint32_t (&bw)[NF / 2],
                                        v8i a_sp, v8i a_dn, uint32_t ssp, uint32_t sdn, int lane) {
  const int half = lane >> 5, col = lane & 31;
  v8i b[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
    b[f] = as_operand(*reinterpret_cast<const uint4*>(lds_w + (f * 32 + col) * kLdsStride + 32 * SUB + 16 * half));
  // backbone products first, then the residual products into the same
  // accumulators: consecutive MFMAs never depend on each other.  The weight
  // scale of fragment f is byte 2 (f & 1) + SUB of word f / 2.
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    if (f & 1) acc[f] = mfma_fp4<2 * SUB, 2 + SUB>(a_sp, b[f], acc[f], ssp, bw[f >> 1]);
    else       acc[f] = mfma_fp4<2 * SUB, SUB>(a_sp, b[f], acc[f], ssp, bw[f >> 1]);
  }
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    if (f & 1) acc[f] = mfma_fp4<2 * SUB, 2 + SUB>(a_dn, b[f], acc[f], sdn, bw[f >> 1]);
    else       acc[f] = mfma_fp4<2 * SUB, SUB>(a_dn, b[f], acc[f], sdn, bw[f >> 1]);
  }
}

// One K step: expand the backbone of both sub-steps, then 2 x NF backbone and
// 2 x NF residual MFMAs against the staged weight tile.
template <int NF, int PAT>
__device__ __forceinline__ void step_mx(v16f (&acc)[NF], const AStep& cur, const uint8_t* lw, const uint8_t* ls,
                                        int lane) {
  static_assert(NF == 8 || NF == 4, "scale record is read as 16 or 8 bytes");
  const int half = lane >> 5, col = lane & 31;
  uint32_t bw[NF / 2];
  if (NF == 8) {
    const uint4 q = *reinterpret_cast<const uint4*>(ls + (2 * col + half) * (2 * NF));
    bw[0] = q.x; bw[1] = q.y; bw[NF / 2 > 2 ? 2 : 0] = q.z; bw[NF / 2 > 3 ? 3 : 0] = q.w;
  } else {
    const uint2 q = *reinterpret_cast<const uint2*>(ls + (2 * col + half) * (2 * NF));
    bw[0] = q.x; bw[NF / 2 > 1 ? 1 : 0] = q.y;
  }
  // op_sel 0 / 2 then picks block 4 ks + half (sub-step 0) / 4 ks + 2 + half (sub-step 1)
  const uint32_t ssp = cur.ssp >> (8 * half), sdn = cur.sdn >> (8 * half);
  {
    const v8i a_sp = as_operand(expand_block<PAT>(cur.spc[0], cur.spm[0]));
    mma_sub<0, NF>(acc, lw, bw, a_sp, as_operand(cur.dn[0]), ssp, sdn, lane);
  }
  {
    const v8i a_sp = as_operand(expand_block<PAT>(cur.spc[1], cur.spm[1]));
    mma_sub<1, NF>(acc, lw, bw, a_sp, as_operand(cur.dn[1]), ssp, sdn, lane);
  }
}

template <typename OutT>
__device__ __forceinline__ void store_out(OutT* p, float v);
template <>
__device__ __forceinline__ void store_out<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store_out<uint16_t>(uint16_t* p, float v) { *p = f32_to_bf16_rne(v); }
template <>
__device__ __forceinline__ void store_out<_Float16>(_Float16* p, float v) { *p = (_Float16)v; }

// One 128 x (32 NF) output tile.  Rows of the tile are output rows
// [row_lo, row_lo + 128) clipped at row_hi; the activation row of output row
// i is row_index[i] when row_index is given, else i - out_base + act_base.
template <int NF, int PAT, bool SCALE_DW, typename OutT>
__device__ __forceinline__ void tile_mx(const uint8_t* sp_codes, const uint8_t* sp_meta, const uint8_t* sp_scale,
                                        const uint8_t* dn_codes, const uint8_t* dn_scale, const int32_t* row_index,
                                        int64_t act_rows, int64_t row_lo, int64_t row_hi, const uint8_t* wc,
                                        const uint8_t* ws, int n0,
                                        int N, int K, OutT* Y, int64_t ldy, uint8_t* lds_w, uint8_t* lds_s) {
  constexpr int BN = 32 * NF;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5;
  const int nblk = K / 32, nks = (K + kBK - 1) / kBK;

  int64_t orow = row_lo + wave * 32 + (lane & 31);
  if (orow >= row_hi) orow = row_hi - 1;   // clamp: loads stay in bounds, stores are masked
  ARow a;
  a.r = row_index ? (int64_t)row_index[orow] : orow;
  a.R = act_rows;
  a.dn = dn_codes;
  a.spc = sp_codes;
  a.spm = sp_meta;
  a.dns = dn_scale;
  a.sps = sp_scale;

  v16f acc[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[f][r] = 0.0f;

  // Software pipeline over K steps, unrolled by two so that the two
  // activation register sets alternate by position instead of being copied.
  // Step ks computes from LDS buffer ks & 1 and register set ks & 1; after
  // its MFMAs the weight tile of step ks+1 (loaded one step earlier) goes to
  // the other LDS buffer and the loads of step ks+2 are issued, so every
  // global load has one full step of MFMA work to arrive.  Loads past the
  // last step re-read the last step (clamped) and are never used.
  AStep a0, a1;
  WStep<NF> wn;
  const int last = nks - 1;
  load_w<NF, SCALE_DW>(wn, wc, ws, n0, N, K, 0, nblk);
  load_a<SCALE_DW>(a0, a, 0, half, nblk, K);
  store_w<NF>(wn, lds_w, lds_s);
  load_w<NF, SCALE_DW>(wn, wc, ws, n0, N, K, min(1, last), nblk);
  load_a<SCALE_DW>(a1, a, min(1, last), half, nblk, K);
  // The scheduling fences keep each phase in place: without them the
  // compiler hoists ALU work on freshly issued loads into the preceding MFMA
  // phase, which then has to wait for those loads.
  constexpr int SREC = 64 * 2 * NF;   // bytes of one buffer's scale records
  int ks = 0;
  for (; ks + 1 < nks; ks += 2) {   // one exit: the accumulators stay in place
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    step_mx<NF, PAT>(acc, a0, lds_w, lds_s, lane);
    __builtin_amdgcn_sched_barrier(0);
    store_w<NF>(wn, lds_w + BN * kLdsStride, lds_s + SREC);
    load_w<NF, SCALE_DW>(wn, wc, ws, n0, N, K, min(ks + 2, last), nblk);
    load_a<SCALE_DW>(a0, a, min(ks + 2, last), half, nblk, K);
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    step_mx<NF, PAT>(acc, a1, lds_w + BN * kLdsStride, lds_s + SREC, lane);
    __builtin_amdgcn_sched_barrier(0);
    store_w<NF>(wn, lds_w, lds_s);
    load_w<NF, SCALE_DW>(wn, wc, ws, n0, N, K, min(ks + 3, last), nblk);
    load_a<SCALE_DW>(a1, a, min(ks + 3, last), half, nblk, K);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (ks < nks) {   // odd number of steps: the last one is in buffer 0 / set 0
    __syncthreads();
    step_mx<NF, PAT>(acc, a0, lds_w, lds_s, lane);
  }

#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int col = n0 + f * 32 + (lane & 31);
    if (col >= N) continue;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t row = row_lo + wave * 32 + 8 * (r / 4) + 4 * half + (r % 4);
      if (row < row_hi) store_out<OutT>(Y + row * ldy + col, acc[f][r]);
    }
  }
}

// ---------------------------------------------------------------------------
// Interleaved main loop (K a multiple of 128, 256 output columns)
// ---------------------------------------------------------------------------
//
// With one wavefront per SIMD the matrix core idles whenever the wavefront
// issues anything but MFMAs, unless that work sits between MFMAs it does not
// feed and is short enough (a wave64 VALU instruction takes 4 cycles, one
// FP4 32x32x64 MFMA 32) to finish before the next MFMA may issue.  Each K step
// therefore runs its 32 MFMAs as fixed slots and spreads the preparation of
// later steps thinly between them: the weight reads of its second sub-step,
// the expansion of the next step's backbone (one 16-bit piece, ~8 VALU, per
// slot), the copy of its residual operand, the LDS store of the weight tile
// two steps ahead and the reads of the next step's first weight operands.
// The weight tile goes through three LDS stages, so the tile of step k+1 is
// published one barrier before step k ends and its first operands are already
// in registers when step k+1 begins.  The global loads of later steps (the
// weights three steps ahead, the activations two steps ahead) go out in six
// parts behind the first six MFMAs rather than as one block before the first:
// measured on the Llama prefill shapes, a block of ~10 loads and their
// address arithmetic ahead of every step left the matrix core idle, and
// spreading them took the three GEMMs from ~450 to ~420-430 us.
// Scheduling fences keep every slot in place.

struct AOps {        // MFMA-ready activation operands of one K step
  uint4 sp[2], dn[2];
  uint32_t ssp, sdn; // E8M0 scale dwords shifted to this lane's half
};

#define SHARQ_FENCE() __builtin_amdgcn_sched_barrier(0)

constexpr int kStageW = 256 * kLdsStride;        // weight codes of one stage
constexpr int kStageBytes = kStageW + 64 * 16;   // + the 64 scale records

// 4:8 expansion through a table.  For a keep mask m, entry m holds two
// v_perm selectors: byte i of the first picks the code for position 2 i (its
// index among the kept codes, or 0x0C = zero if position 2 i is dropped), the
// second the code for position 2 i + 1.  The group's four codes are spread to
// bytes, permuted twice (once shifted into the high nibbles) and OR-ed.
__device__ __forceinline__ uint2 lut48_entry(uint32_t m) {
  uint32_t se = 0u, so = 0u, idx = 0u;
#pragma unroll
  for (int p = 0; p < 8; ++p) {
    uint32_t sel = 0x0Cu;
    if ((m >> p) & 1u) sel = idx++;
    if (p & 1) so |= sel << (8 * (p >> 1));
    else se |= sel << (8 * (p >> 1));
  }
  return make_uint2(se, so);
}

__device__ __forceinline__ uint32_t expand48_lut(uint32_t c16, uint2 sel) {
  uint32_t x = (c16 | (c16 << 8)) & 0x00FF00FFu;   // bytes 0, 2: code pairs (0, 1), (2, 3)
  x = (x | (x << 4)) & 0x0F0F0F0Fu;                 // byte i: code i
  return __builtin_amdgcn_perm(0u, x, sel.x) | __builtin_amdgcn_perm(0u, x << 4, sel.y);
}

// Fill a workgroup's 256-entry table (one entry per thread); the caller
// synchronizes before the first use.
__device__ __forceinline__ void lut48_fill(uint2* lut) {
  if (threadIdx.x < 256) lut[threadIdx.x] = lut48_entry(threadIdx.x);
}


// Piece Q (0..15) of the next step's expanded backbone: block Q / 8, output
// dword (Q % 8) / 2, 16-bit half Q % 2 (returned in place within the dword).
template <int PAT, int Q>
__device__ __forceinline__ uint32_t exp_piece(const AStep& r) {
  constexpr int B = Q / 8, D = (Q % 8) / 2, H = Q % 2;
  const uint2 c = r.spc[B];
  const uint32_t meta = r.spm[B];
  if (PAT == 24) {
    constexpr int G = 2 * D + H;   // group of 4 positions
    const uint32_t cw = G < 4 ? c.x : c.y;
    const uint32_t byte = (cw >> (8 * (G & 3))) & 0xFFu;
    const uint32_t nib = (meta >> (4 * G)) & 0xFu;
    return ((byte & 0xFu) << (4 * (nib & 3u) + 16 * H)) | ((byte >> 4) << (4 * (nib >> 2) + 16 * H));
  } else {
    constexpr int G = D;           // group of 8 positions, half H of it
    const uint32_t cw = G < 2 ? c.x : c.y;
    uint32_t c16 = (cw >> (16 * (G & 1))) & 0xFFFFu;
    const uint32_t mask = (meta >> (8 * G)) & 0xFFu;
    if (H == 1) c16 >>= 4 * __builtin_popcount(mask & 0xFu);
    uint32_t out = 0u;
#pragma unroll
    for (int p = 4 * H; p < 4 * H + 4; ++p) {
      if ((mask >> p) & 1u) {
        out |= (c16 & 0xFu) << (4 * p);
        c16 >>= 4;
      }
    }
    return out;
  }
}

template <int PAT, int Q>
__device__ __forceinline__ void put_piece(AOps& o, const AStep& r, const uint2 (&sel)[8]) {
  if (PAT == 0) return;   // the backbone arrives dense
  constexpr int B = Q / 8, D = (Q % 8) / 2, H = Q % 2;
  uint32_t& d = D == 0 ? o.sp[B].x : D == 1 ? o.sp[B].y : D == 2 ? o.sp[B].z : o.sp[B].w;
  if (PAT == 48) {
    // a whole group (output dword) per even piece, from its table entry
    if (H == 0) {
      const uint32_t cw = D < 2 ? r.spc[B].x : r.spc[B].y;
      d = expand48_lut((cw >> (16 * (D & 1))) & 0xFFFFu, sel[4 * B + D]);
    }
  } else {
    const uint32_t v = exp_piece<PAT, Q>(r);
    d = H == 0 ? v : (d | v);
  }
}

// The weight is the MFMA's first operand and the activation its second, so
// the accumulator is the transposed tile: lane l holds activation row
// l % 32 and, in element r, output column 8 (r / 4) + 4 (l / 32) + r % 4 of
// the fragment -- four consecutive columns per group of four elements.
template <int SUB, int F, int NF>
__device__ __forceinline__ void mma_sp(v16f (&acc)[NF], const AOps& a, const uint4 (&b)[NF],
                                       const uint32_t (&bw)[NF / 2]) {
  acc[F] = mfma_fp4<(F & 1) ? 2 + SUB : SUB, SUB>(as_operand(b[F]), as_operand(a.sp[SUB]), acc[F], bw[F >> 1],
                                                 a.ssp);
}

template <int SUB, int F, int NF>
__device__ __forceinline__ void mma_dn(v16f (&acc)[NF], const AOps& a, const uint4 (&b)[NF],
                                       const uint32_t (&bw)[NF / 2]) {
  acc[F] = mfma_fp4<(F & 1) ? 2 + SUB : SUB, SUB>(as_operand(b[F]), as_operand(a.dn[SUB]), acc[F], bw[F >> 1],
                                                 a.sdn);
}

template <typename OutT>
struct Vec4Out;
template <>
struct Vec4Out<float> {
  static __device__ __forceinline__ void put(float* p, float a, float b, float c, float d) {
    *reinterpret_cast<float4*>(p) = make_float4(a, b, c, d);
  }
  static constexpr int kAlign = 16;
};
template <>
struct Vec4Out<uint16_t> {
  static __device__ __forceinline__ void put(uint16_t* p, float a, float b, float c, float d) {
    // v_cvt_pk_bf16_f32: two round-to-nearest-even conversions per instruction
    typedef __bf16 bf4 __attribute__((ext_vector_type(4)));
    bf4 v;
    v[0] = (__bf16)a; v[1] = (__bf16)b; v[2] = (__bf16)c; v[3] = (__bf16)d;
    *reinterpret_cast<bf4*>(p) = v;
  }
  static constexpr int kAlign = 8;
};
template <>
struct Vec4Out<_Float16> {
  static __device__ __forceinline__ void put(_Float16* p, float a, float b, float c, float d) {
    typedef _Float16 h4 __attribute__((ext_vector_type(4)));
    h4 v;
    v[0] = (_Float16)a; v[1] = (_Float16)b; v[2] = (_Float16)c; v[3] = (_Float16)d;
    *reinterpret_cast<h4*>(p) = v;
  }
  static constexpr int kAlign = 8;
};

template <int SUB, int F0, int F1, int NB>
__device__ __forceinline__ void read_b(uint4 (&b)[NB], const uint8_t* lw, int lane) {
  const int half = lane >> 5, col = lane & 31;
#pragma unroll
  for (int f = F0; f < F1; ++f)
    b[f] = *reinterpret_cast<const uint4*>(lw + (f * 32 + col) * kLdsStride + 32 * half + 16 * SUB);
}

__device__ __forceinline__ void read_bw(uint32_t (&bw)[4], const uint8_t* stage, int lane) {
  const int half = lane >> 5, col = lane & 31;
  const uint4 q = *reinterpret_cast<const uint4*>(stage + kStageW + (2 * col + half) * 16);
  bw[0] = q.x; bw[1] = q.y; bw[2] = q.z; bw[3] = q.w;
}

// half tiles (fragments 0-3): the first 8 bytes of the record
__device__ __forceinline__ void read_bw(uint32_t (&bw)[2], const uint8_t* stage, int lane) {
  const int half = lane >> 5, col = lane & 31;
  const uint2 q = *reinterpret_cast<const uint2*>(stage + kStageW + (2 * col + half) * 16);
  bw[0] = q.x; bw[1] = q.y;
}

// One K step k.  In: b0 / bw = sub-step 0 weight operands and scale records
// of step k (read from stage `cur`); ops = expanded activations of step k.
// Out: b0 / bwn = those of step k+1 (from stage `nxt`); opsn.sp and scales =
// expansion of raw (step k+1; its residual codes are loaded into opsn.dn by
// `issue`); wst (step k+2) stored to stage `wr`.  issue(part) issues part
// 0-5 of the step's global loads (a std::integral_constant argument).
// SPR = 0: the six parts go out behind the first six MFMAs; SPR = 1: spread
// over the whole step, two slots of each group of eight apart (the schedule of
// the row-gathering grouped GEMM, whose scattered activation rows make each
// load slower to issue; for contiguous rows the burst is faster).
template <int PAT, int SPR = 0, class Issue>
__device__ __forceinline__ void step5(v16f (&acc)[8], const AOps& ops, uint4 (&b0)[8], const uint32_t (&bw)[4],
                                      uint32_t (&bwn)[4], const uint8_t* cur, const uint8_t* nxt, uint8_t* wr,
                                      AOps& opsn, const AStep& raw, const WStep<8>& wst, int lane, Issue issue,
                                      const uint2* lut) {
  const int half = lane >> 5, tid = threadIdx.x;
  uint4 b1[8];
  uint2 sel[8];
  if (PAT == 48) {   // table entries of the next step's eight 4:8 groups
#pragma unroll
    for (int i = 0; i < 8; ++i) sel[i] = lut[(raw.spm[i >> 2] >> (8 * (i & 3))) & 0xFFu];
  }
  // LDS traffic is spread at about one instruction per slot (a 1 KB
  // wavefront access keeps the LDS busy for several MFMA-lengths when four
  // wavefronts burst together); VALU work stays under ~8 instructions per slot.
  // ---- sub-step 0, backbone: second sub-step's weight operands; the
  // global loads of later steps go out in six parts behind the first MFMAs
  mma_sp<0, 0>(acc, ops, b0, bw); issue(std::integral_constant<int, 0>()); read_b<1, 0, 1>(b1, cur, lane);
  put_piece<PAT, 0>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<0, 1>(acc, ops, b0, bw);
  if constexpr (SPR == 0) issue(std::integral_constant<int, 1>());
  read_b<1, 1, 2>(b1, cur, lane);
  SHARQ_FENCE();
  mma_sp<0, 2>(acc, ops, b0, bw);
  if constexpr (SPR == 0) issue(std::integral_constant<int, 2>());
  read_b<1, 2, 3>(b1, cur, lane);
  put_piece<PAT, 1>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<0, 3>(acc, ops, b0, bw);
  if constexpr (SPR == 0) issue(std::integral_constant<int, 3>());
  read_b<1, 3, 4>(b1, cur, lane);
  SHARQ_FENCE();
  mma_sp<0, 4>(acc, ops, b0, bw);
  if constexpr (SPR == 0) issue(std::integral_constant<int, 4>());
  read_b<1, 4, 5>(b1, cur, lane);
  put_piece<PAT, 2>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<0, 5>(acc, ops, b0, bw);
  if constexpr (SPR == 0) issue(std::integral_constant<int, 5>());
  else issue(std::integral_constant<int, 1>());
  read_b<1, 5, 6>(b1, cur, lane);
  SHARQ_FENCE();
  mma_sp<0, 6>(acc, ops, b0, bw); read_b<1, 6, 7>(b1, cur, lane); put_piece<PAT, 3>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<0, 7>(acc, ops, b0, bw); read_b<1, 7, 8>(b1, cur, lane); SHARQ_FENCE();
  // ---- sub-step 0, residual: the weight tile two steps ahead to LDS
  mma_dn<0, 0>(acc, ops, b0, bw); put_piece<PAT, 4>(opsn, raw, sel); SHARQ_FENCE();
  mma_dn<0, 1>(acc, ops, b0, bw);
  *reinterpret_cast<uint4*>(wr + (tid >> 2) * kLdsStride + 16 * (tid & 3)) = wst.q[0];
  SHARQ_FENCE();
  mma_dn<0, 2>(acc, ops, b0, bw); put_piece<PAT, 5>(opsn, raw, sel);
  if constexpr (SPR == 1) issue(std::integral_constant<int, 2>());
  SHARQ_FENCE();
  mma_dn<0, 3>(acc, ops, b0, bw);
  *reinterpret_cast<uint4*>(wr + ((tid + 256) >> 2) * kLdsStride + 16 * (tid & 3)) = wst.q[1];
  SHARQ_FENCE();
  mma_dn<0, 4>(acc, ops, b0, bw); put_piece<PAT, 6>(opsn, raw, sel); SHARQ_FENCE();
  mma_dn<0, 5>(acc, ops, b0, bw);
  *reinterpret_cast<uint4*>(wr + ((tid + 512) >> 2) * kLdsStride + 16 * (tid & 3)) = wst.q[2];
  SHARQ_FENCE();
  mma_dn<0, 6>(acc, ops, b0, bw); put_piece<PAT, 7>(opsn, raw, sel);
  if constexpr (SPR == 1) issue(std::integral_constant<int, 3>());
  SHARQ_FENCE();
  mma_dn<0, 7>(acc, ops, b0, bw);
  *reinterpret_cast<uint4*>(wr + ((tid + 768) >> 2) * kLdsStride + 16 * (tid & 3)) = wst.q[3];
  SHARQ_FENCE();
  // ---- sub-step 1, backbone: weight scales, then the next step's operands
  mma_sp<1, 0>(acc, ops, b1, bw); put_piece<PAT, 8>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<1, 1>(acc, ops, b1, bw);
  {
    const int f = tid >> 5, c = tid & 31;
    // record (c, h) byte 2 (f & 1) + sub <- block 2 h + sub of weight row 32 f + c
    *reinterpret_cast<uint16_t*>(wr + kStageW + (2 * c + 0) * 16 + 2 * f) = (uint16_t)wst.s;
    *reinterpret_cast<uint16_t*>(wr + kStageW + (2 * c + 1) * 16 + 2 * f) = (uint16_t)(wst.s >> 16);
  }
  SHARQ_FENCE();
  mma_sp<1, 2>(acc, ops, b1, bw); put_piece<PAT, 9>(opsn, raw, sel);
  if constexpr (SPR == 1) issue(std::integral_constant<int, 4>());
  SHARQ_FENCE();
  mma_sp<1, 3>(acc, ops, b1, bw); read_b<0, 0, 1>(b0, nxt, lane); SHARQ_FENCE();
  mma_sp<1, 4>(acc, ops, b1, bw); put_piece<PAT, 10>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<1, 5>(acc, ops, b1, bw); read_b<0, 1, 2>(b0, nxt, lane); SHARQ_FENCE();
  mma_sp<1, 6>(acc, ops, b1, bw); put_piece<PAT, 11>(opsn, raw, sel);
  if constexpr (SPR == 1) issue(std::integral_constant<int, 5>());
  SHARQ_FENCE();
  mma_sp<1, 7>(acc, ops, b1, bw); read_b<0, 2, 3>(b0, nxt, lane); SHARQ_FENCE();
  // ---- sub-step 1, residual
  mma_dn<1, 0>(acc, ops, b1, bw); put_piece<PAT, 12>(opsn, raw, sel); read_b<0, 3, 4>(b0, nxt, lane); SHARQ_FENCE();
  mma_dn<1, 1>(acc, ops, b1, bw); read_b<0, 4, 5>(b0, nxt, lane); SHARQ_FENCE();
  mma_dn<1, 2>(acc, ops, b1, bw); put_piece<PAT, 13>(opsn, raw, sel); read_b<0, 5, 6>(b0, nxt, lane); SHARQ_FENCE();
  mma_dn<1, 3>(acc, ops, b1, bw); read_b<0, 6, 7>(b0, nxt, lane); SHARQ_FENCE();
  mma_dn<1, 4>(acc, ops, b1, bw); put_piece<PAT, 14>(opsn, raw, sel); read_b<0, 7, 8>(b0, nxt, lane); SHARQ_FENCE();
  mma_dn<1, 5>(acc, ops, b1, bw); read_bw(bwn, nxt, lane); SHARQ_FENCE();
  mma_dn<1, 6>(acc, ops, b1, bw); put_piece<PAT, 15>(opsn, raw, sel); SHARQ_FENCE();
  mma_dn<1, 7>(acc, ops, b1, bw);
  opsn.ssp = raw.ssp >> (16 * half);
  opsn.sdn = raw.sdn >> (16 * half);
  if (PAT == 0) {
    opsn.sp[0] = raw.spd[0];
    opsn.sp[1] = raw.spd[1];
  }
  SHARQ_FENCE();
}

// The same K step for a half tile (128 output columns, fragments 0-3): 16
// MFMA slots.  The weight stage keeps the full tile's layout with rows 0-127
// (and bytes 0-7 of each scale record) filled, so the operand reads are the
// full tile's; the extra work per slot is about twice as dense.
template <int PAT, class Issue>
__device__ __forceinline__ void step5h(v16f (&acc)[4], const AOps& ops, uint4 (&b0)[4], const uint32_t (&bw)[2],
                                       uint32_t (&bwn)[2], const uint8_t* cur, const uint8_t* nxt, uint8_t* wr,
                                       AOps& opsn, const AStep& raw, const WStep<4>& wst, int lane, Issue issue,
                                       const uint2* lut) {
  const int half = lane >> 5, tid = threadIdx.x;
  uint4 b1[4];
  uint2 sel[8];
  if (PAT == 48) {
#pragma unroll
    for (int i = 0; i < 8; ++i) sel[i] = lut[(raw.spm[i >> 2] >> (8 * (i & 3))) & 0xFFu];
  }
  // ---- sub-step 0: the second sub-step's weight operands and the global
  // loads of later steps, then the weight tile two steps ahead to LDS
  mma_sp<0, 0>(acc, ops, b0, bw); issue(std::integral_constant<int, 0>()); read_b<1, 0, 1>(b1, cur, lane);
  put_piece<PAT, 0>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<0, 1>(acc, ops, b0, bw); issue(std::integral_constant<int, 1>()); read_b<1, 1, 2>(b1, cur, lane);
  put_piece<PAT, 1>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<0, 2>(acc, ops, b0, bw); issue(std::integral_constant<int, 2>()); read_b<1, 2, 3>(b1, cur, lane);
  put_piece<PAT, 2>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<0, 3>(acc, ops, b0, bw); issue(std::integral_constant<int, 3>()); read_b<1, 3, 4>(b1, cur, lane);
  put_piece<PAT, 3>(opsn, raw, sel); SHARQ_FENCE();
  mma_dn<0, 0>(acc, ops, b0, bw); issue(std::integral_constant<int, 4>()); put_piece<PAT, 4>(opsn, raw, sel);
  *reinterpret_cast<uint4*>(wr + (tid >> 2) * kLdsStride + 16 * (tid & 3)) = wst.q[0];
  SHARQ_FENCE();
  mma_dn<0, 1>(acc, ops, b0, bw); issue(std::integral_constant<int, 5>()); put_piece<PAT, 5>(opsn, raw, sel);
  *reinterpret_cast<uint4*>(wr + ((tid + 256) >> 2) * kLdsStride + 16 * (tid & 3)) = wst.q[1];
  SHARQ_FENCE();
  mma_dn<0, 2>(acc, ops, b0, bw); put_piece<PAT, 6>(opsn, raw, sel);
  {
    // threads 128-255 hold a copy of column 127's scales and write bytes 8-15
    // of the records, which a half tile never reads: no branch, so the step
    // stays one basic block and the compiler keeps every MFMA in its slot
    const int f = tid >> 5, c = tid & 31;
    *reinterpret_cast<uint16_t*>(wr + kStageW + (2 * c + 0) * 16 + 2 * f) = (uint16_t)wst.s;
    *reinterpret_cast<uint16_t*>(wr + kStageW + (2 * c + 1) * 16 + 2 * f) = (uint16_t)(wst.s >> 16);
  }
  SHARQ_FENCE();
  mma_dn<0, 3>(acc, ops, b0, bw); put_piece<PAT, 7>(opsn, raw, sel); SHARQ_FENCE();
  // ---- sub-step 1: the next step's first operands and scale records
  mma_sp<1, 0>(acc, ops, b1, bw); put_piece<PAT, 8>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<1, 1>(acc, ops, b1, bw); read_b<0, 0, 1>(b0, nxt, lane); put_piece<PAT, 9>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<1, 2>(acc, ops, b1, bw); read_b<0, 1, 2>(b0, nxt, lane); put_piece<PAT, 10>(opsn, raw, sel); SHARQ_FENCE();
  mma_sp<1, 3>(acc, ops, b1, bw); read_b<0, 2, 3>(b0, nxt, lane); put_piece<PAT, 11>(opsn, raw, sel); SHARQ_FENCE();
  mma_dn<1, 0>(acc, ops, b1, bw); read_b<0, 3, 4>(b0, nxt, lane); put_piece<PAT, 12>(opsn, raw, sel); SHARQ_FENCE();
  mma_dn<1, 1>(acc, ops, b1, bw); read_bw(bwn, nxt, lane); put_piece<PAT, 13>(opsn, raw, sel); SHARQ_FENCE();
  mma_dn<1, 2>(acc, ops, b1, bw); put_piece<PAT, 14>(opsn, raw, sel); SHARQ_FENCE();
  mma_dn<1, 3>(acc, ops, b1, bw); put_piece<PAT, 15>(opsn, raw, sel);
  opsn.ssp = raw.ssp >> (16 * half);
  opsn.sdn = raw.sdn >> (16 * half);
  if (PAT == 0) {
    opsn.sp[0] = raw.spd[0];
    opsn.sp[1] = raw.spd[1];
  }
  SHARQ_FENCE();
}

// Residual codes of step ks straight into the operand registers, and the
// backbone codes / metadata / scales of step ks into a raw set (panel-major,
// K a multiple of 128).
// In this loop lane half h takes blocks 2h and 2h+1 of each 128-position
// step (sub-step s uses block 2h + s), so a lane's bytes of every buffer are
// contiguous: 32 bytes of residual codes, 16 of backbone codes, 8 of metadata.
__device__ __forceinline__ void load_a_dn(AOps& o, const ARow& a, int ks, int half) {
  const uint8_t* dn = a.dn + (int64_t)ks * a.R * 64 + a.r * 64 + 32 * half;
  o.dn[0] = *reinterpret_cast<const uint4*>(dn);
  o.dn[1] = *reinterpret_cast<const uint4*>(dn + 16);
}

// PAT 0: a.spc is the dense backbone copy, laid out like the residual codes.
template <int PAT>
__device__ __forceinline__ void load_a_meta(AStep& s, const ARow& a, int ks, int half) {
  const int64_t pr = (int64_t)ks * a.R;
  if (PAT == 0) {
    const uint8_t* sp = a.spc + pr * 64 + a.r * 64 + 32 * half;
    s.spd[0] = *reinterpret_cast<const uint4*>(sp);
    s.spd[1] = *reinterpret_cast<const uint4*>(sp + 16);
  } else {
    const uint4 c = *reinterpret_cast<const uint4*>(a.spc + pr * 32 + a.r * 32 + 16 * half);
    const uint2 m = *reinterpret_cast<const uint2*>(a.spm + pr * 16 + a.r * 16 + 8 * half);
    s.spc[0] = make_uint2(c.x, c.y);
    s.spc[1] = make_uint2(c.z, c.w);
    s.spm[0] = m.x;
    s.spm[1] = m.y;
  }
  s.sdn = *reinterpret_cast<const uint32_t*>(a.dns + pr * 4 + a.r * 4);
  s.ssp = *reinterpret_cast<const uint32_t*>(a.sps + pr * 4 + a.r * 4);
}


// Parts of one K step's global loads (K a multiple of 128), so that the
// interleaved loop can spread them over its MFMA slots: the backbone codes
// (or the dense copy) and the two scale dwords of the activations; two halves
// of the weight codes and the weight scales (load_w's bytes, in parts).
template <int PAT, int P>
__device__ __forceinline__ void load_a_meta_part(AStep& s, const ARow& a, int ks, int half) {
  const int64_t pr = (int64_t)ks * a.R;
  if constexpr (P == 0) {
    if (PAT == 0) {
      const uint8_t* sp = a.spc + pr * 64 + a.r * 64 + 32 * half;
      s.spd[0] = *reinterpret_cast<const uint4*>(sp);
      s.spd[1] = *reinterpret_cast<const uint4*>(sp + 16);
    } else {
      const uint4 c = *reinterpret_cast<const uint4*>(a.spc + pr * 32 + a.r * 32 + 16 * half);
      const uint2 m = *reinterpret_cast<const uint2*>(a.spm + pr * 16 + a.r * 16 + 8 * half);
      s.spc[0] = make_uint2(c.x, c.y);
      s.spc[1] = make_uint2(c.z, c.w);
      s.spm[0] = m.x;
      s.spm[1] = m.y;
    }
  } else {
    s.sdn = *reinterpret_cast<const uint32_t*>(a.dns + pr * 4 + a.r * 4);
    s.ssp = *reinterpret_cast<const uint32_t*>(a.sps + pr * 4 + a.r * 4);
  }
}

template <int NF, int P>
__device__ __forceinline__ void load_w_part(WStep<NF>& w, const uint8_t* wc, const uint8_t* ws, int n0, int N,
                                            int ks) {
  constexpr int BN = 32 * NF;
  const int tid = threadIdx.x;
  const int64_t pn = (int64_t)ks * N;
  if constexpr (P < 2) {
#pragma unroll
    for (int j = P * NF / 4; j < (P + 1) * NF / 4; ++j) {
      const int c = tid + 256 * j;
      const int row = c >> 2, part = c & 3;
      const int n = min(n0 + row, N - 1);
      w.q[j] = *reinterpret_cast<const uint4*>(wc + pn * 64 + (int64_t)n * 64 + 16 * part);
    }
  } else {
    // In a half tile threads BN..255 load column BN - 1's scales again: their
    // copy lands in record bytes that a half tile never reads.  Selecting 0
    // for them instead would make the value depend on the load at issue time,
    // and the wait for it (the newest load) drained every load in flight once
    // per step: 57.5 -> 53.5 us on the Llama qkv shape, whose last round runs
    // as half tiles.
    const int n = min(n0 + (BN >= 256 ? tid : min(tid, BN - 1)), N - 1);
    w.s = *reinterpret_cast<const uint32_t*>(ws + pn * 4 + (int64_t)n * 4);
  }
}

template <int NF>
__device__ __forceinline__ void store_w_stage(const WStep<NF>& w, uint8_t* stage) {
  const int tid = threadIdx.x;
#pragma unroll
  for (int j = 0; j < NF / 2; ++j) {
    const int c = tid + 256 * j;
    *reinterpret_cast<uint4*>(stage + (c >> 2) * kLdsStride + 16 * (c & 3)) = w.q[j];
  }
  if (NF == 8 || tid < 32 * NF) {
    const int f = tid >> 5, c = tid & 31;
    *reinterpret_cast<uint16_t*>(stage + kStageW + (2 * c + 0) * 16 + 2 * f) = (uint16_t)w.s;
    *reinterpret_cast<uint16_t*>(stage + kStageW + (2 * c + 1) * 16 + 2 * f) = (uint16_t)(w.s >> 16);
  }
}

// Epilogue of a wavefront's 32 x 256 block of 2-byte outputs through LDS.
// In the accumulator layout a lane holds 8-byte pieces of one output row, so
// direct stores put 32 scattered 16-byte pieces in every instruction (rows
// are N outputs apart); measured on the Llama prefill shapes this cost about
// 5 us per round of tiles.  Here the block is staged in LDS and read back
// along rows: each store instruction then writes two whole 512-byte row
// segments.  The wavefront owns its LDS region, and its LDS accesses execute
// in order, so no barrier is needed inside.
// A value that is the same in every lane, read from the first active one.
__device__ __forceinline__ int64_t uniform64(int64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Fourth dword of a raw buffer resource (no stride, no swizzle, 32-bit
// data format: the range check is on the byte offset).
constexpr int kBufferWord3 = 0x00020000;
typedef uint32_t v4u32_t __attribute__((ext_vector_type(4)));

constexpr int kEpiStride = 528;            // bytes per staged row: 512 + 16 (spreads rows over banks)
constexpr int kEpiWave = 32 * kEpiStride;  // one wavefront's region
constexpr int kTileLds = 4 * kEpiWave > 3 * kStageBytes ? 4 * kEpiWave : 3 * kStageBytes;
constexpr int kPersistLds = 3 * kStageBytes + 4 * kEpiWave;   // stages and epilogue apart: 129 KB

template <typename OutT, int NF>
__device__ __forceinline__ void store_tile_lds(const v16f (&acc)[NF], OutT* Y, int64_t ldy, int64_t row0,
                                               int64_t row_hi, int n0, int N, uint8_t* buf, int lane) {
  // a staged row is 64 NF bytes (+16); 4 NF lanes read it back, 16 / NF rows per instruction
  constexpr int stride = 64 * NF + 16, lpr = 4 * NF, rpi = 64 / lpr;
  const int r = lane & 31, half = lane >> 5;
#pragma unroll
  for (int f = 0; f < NF; ++f) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      Vec4Out<OutT>::put(reinterpret_cast<OutT*>(buf + r * stride + (32 * f + 8 * g + 4 * half) * 2),
                         acc[f][4 * g], acc[f][4 * g + 1], acc[f][4 * g + 2], acc[f][4 * g + 3]);
    }
  }
  // every read back first: a store under a per-row condition would take its
  // read into its own branch and wait for it there, one LDS round trip per
  // store
  constexpr int kReads = 32 / rpi;
  uint4 v[kReads];
#pragma unroll
  for (int i = 0; i < kReads; ++i)
    v[i] = *reinterpret_cast<const uint4*>(buf + (rpi * i + lane / lpr) * stride + (lane % lpr) * 16);
  // row0 and row_hi are the same in every lane; the compiler cannot see it,
  // and a buffer resource held in vector registers would cost a loop over
  // lanes around every store
  row0 = uniform64(row0);
  row_hi = uniform64(row_hi);
  const int64_t rows = row_hi - row0 < 32 ? row_hi - row0 : 32;   // the wavefront's rows in the tile
  if (rows <= 0) return;
  const int64_t span = rows * ldy * (int64_t)sizeof(OutT);
  const int ch = lane % lpr, col = n0 + 8 * ch;
  if (span <= (int64_t)1 << 30) {
    // Unconditional buffer stores over a range of exactly the wavefront's
    // rows: the range check drops a store to a row past the tile, and a
    // column past N gets an offset (2^31 - 16) past any such range.
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(Y + row0 * ldy, (short)0, (int)span,
                                                                        kBufferWord3);
#pragma unroll
    for (int i = 0; i < kReads; ++i) {
      const int rr = rpi * i + lane / lpr;
      const int off = col < N ? (int)(((int64_t)rr * ldy + col) * (int64_t)sizeof(OutT)) : 0x7FFFFFF0;
      v4u32_t q;
      q[0] = v[i].x; q[1] = v[i].y; q[2] = v[i].z; q[3] = v[i].w;
      __builtin_amdgcn_raw_buffer_store_b128(q, rs, off, 0, 0);
    }
  } else {
#pragma unroll
    for (int i = 0; i < kReads; ++i) {
      const int rr = rpi * i + lane / lpr;
      if (rr < rows && col < N) *reinterpret_cast<uint4*>(Y + (row0 + rr) * ldy + col) = v[i];
    }
  }
}

// One K step of a full (NF = 8) or half (NF = 4) tile; SPR: the load
// schedule of step5.
template <int PAT, int SPR = 0, int NF, class Issue>
__device__ __forceinline__ void step_il(v16f (&acc)[NF], const AOps& ops, uint4 (&b0)[NF],
                                        const uint32_t (&bw)[NF / 2], uint32_t (&bwn)[NF / 2], const uint8_t* cur,
                                        const uint8_t* nxt, uint8_t* wr, AOps& opsn, const AStep& raw,
                                        const WStep<NF>& wst, int lane, Issue issue, const uint2* lut) {
  if constexpr (NF == 8)
    step5<PAT, SPR>(acc, ops, b0, bw, bwn, cur, nxt, wr, opsn, raw, wst, lane, issue, lut);
  else
    step5h<PAT>(acc, ops, b0, bw, bwn, cur, nxt, wr, opsn, raw, wst, lane, issue, lut);
}

// The register sets of the interleaved pipeline.  They rotate with period
// three, so the main loop is unrolled by three and the LDS stages are fixed
// per unrolled step.  Invariant at the start of step k (sets indexed by
// k mod 3): stages k, k+1 hold W(k), W(k+1); b0 / bw hold step k's first
// weight operands; o[k] is complete; o[k+1].dn = residual codes of step k+1
// (in flight); r[k+1], r[k+2] = raw backbone data of steps k+1, k+2; w[k+2],
// w[k] = raw W(k+2), W(k+3).  Step k loads the residual codes of step k+2, the
// raw backbone of step k+3 and W(k+4): every load has two full steps to
// arrive.  Loads past the last step re-read it (clamped) and their results
// are never used.
template <int NF>
struct IlSets {
  AStep r0, r1, r2;
  WStep<NF> w0, w1, w2;
  AOps o0, o1, o2;
};

// A tile's first global loads: W(0..2), the residual codes of steps 0 and 1,
// the raw backbone of steps 0..2.  They touch no LDS, so a persistent loop can
// issue them for its next tile before the current tile's output stores.
template <int PAT, int NF>
__device__ __forceinline__ void il_issue(IlSets<NF>& p, const ARow& a, const uint8_t* wc, const uint8_t* ws,
                                         int n0, int N, int K, int half) {
  const int nblk = K / 32, last = K / kBK - 1;
  const auto cl = [&](int k) { return k < last ? k : last; };
  load_w<NF, true>(p.w0, wc, ws, n0, N, K, 0, nblk);
  load_a_meta<PAT>(p.r0, a, 0, half);
  load_a_dn(p.o0, a, 0, half);
  load_w<NF, true>(p.w1, wc, ws, n0, N, K, cl(1), nblk);
  load_a_dn(p.o1, a, cl(1), half);
  load_a_meta<PAT>(p.r1, a, cl(1), half);
  load_a_meta<PAT>(p.r2, a, cl(2), half);
  load_w<NF, true>(p.w2, wc, ws, n0, N, K, cl(2), nblk);
}

// The rest of a tile's prologue: W(0), W(1) into stages 0 and 1, step 0's
// backbone operands, the load of W(3), and step 0's first weight operands.
// The stages must be free (a barrier after the previous tile's last step).
template <int PAT, int NF>
__device__ __forceinline__ void il_start(IlSets<NF>& p, const uint8_t* wc, const uint8_t* ws, int n0, int N,
                                         int K, uint8_t* lds, uint4 (&b0)[NF], uint32_t (&bwa)[NF / 2], int lane,
                                         int half) {
  const int nblk = K / 32, last = K / kBK - 1;
  store_w_stage(p.w0, lds);
  store_w_stage(p.w1, lds + kStageBytes);
  if (PAT == 0) {
    p.o0.sp[0] = p.r0.spd[0];
    p.o0.sp[1] = p.r0.spd[1];
  } else {
    p.o0.sp[0] = expand_block<PAT>(p.r0.spc[0], p.r0.spm[0]);
    p.o0.sp[1] = expand_block<PAT>(p.r0.spc[1], p.r0.spm[1]);
  }
  p.o0.ssp = p.r0.ssp >> (16 * half);
  p.o0.sdn = p.r0.sdn >> (16 * half);
  load_w<NF, true>(p.w0, wc, ws, n0, N, K, 3 < last ? 3 : last, nblk);
  __syncthreads();
  read_bw(bwa, lds, lane);
  read_b<0, 0, NF>(b0, lds, lane);
}

// Every K step of a started tile into acc.
template <int PAT, int NF, int SPR = 0>
__device__ __forceinline__ void il_main(v16f (&acc)[NF], IlSets<NF>& p, uint4 (&b0)[NF], uint32_t (&bwa)[NF / 2],
                                        const ARow& a, const uint8_t* wc, const uint8_t* ws, int n0, int N, int K,
                                        uint8_t* lds, int lane, int half, const uint2* lut) {
  const int nks = K / kBK, last = nks - 1;
  const auto cl = [&](int k) { return k < last ? k : last; };
  uint8_t* const st0 = lds;
  uint8_t* const st1 = lds + kStageBytes;
  uint8_t* const st2 = lds + 2 * kStageBytes;
  uint32_t bwb[NF / 2];
  int ks = 0;
  for (; ks + 2 < nks; ks += 3) {
    step_il<PAT, SPR>(acc, p.o0, b0, bwa, bwb, st0, st1, st2, p.o1, p.r1, p.w2, lane, [&](auto part) {
      constexpr int P = decltype(part)::value;
      if constexpr (P == 0) load_a_dn(p.o2, a, cl(ks + 2), half);
      else if constexpr (P == 1) load_a_meta_part<PAT, 0>(p.r0, a, cl(ks + 3), half);
      else if constexpr (P == 2) load_a_meta_part<PAT, 1>(p.r0, a, cl(ks + 3), half);
      else load_w_part<NF, P - 3>(p.w1, wc, ws, n0, N, cl(ks + 4));
    }, lut);
    __syncthreads();
    step_il<PAT, SPR>(acc, p.o1, b0, bwb, bwa, st1, st2, st0, p.o2, p.r2, p.w0, lane, [&](auto part) {
      constexpr int P = decltype(part)::value;
      if constexpr (P == 0) load_a_dn(p.o0, a, cl(ks + 3), half);
      else if constexpr (P == 1) load_a_meta_part<PAT, 0>(p.r1, a, cl(ks + 4), half);
      else if constexpr (P == 2) load_a_meta_part<PAT, 1>(p.r1, a, cl(ks + 4), half);
      else load_w_part<NF, P - 3>(p.w2, wc, ws, n0, N, cl(ks + 5));
    }, lut);
    __syncthreads();
    step_il<PAT, SPR>(acc, p.o2, b0, bwa, bwb, st2, st0, st1, p.o0, p.r0, p.w1, lane, [&](auto part) {
      constexpr int P = decltype(part)::value;
      if constexpr (P == 0) load_a_dn(p.o1, a, cl(ks + 4), half);
      else if constexpr (P == 1) load_a_meta_part<PAT, 0>(p.r2, a, cl(ks + 5), half);
      else if constexpr (P == 2) load_a_meta_part<PAT, 1>(p.r2, a, cl(ks + 5), half);
      else load_w_part<NF, P - 3>(p.w0, wc, ws, n0, N, cl(ks + 6));
    }, lut);
    __syncthreads();
    // bw alternates with period two: after three steps the roles swap
#pragma unroll
    for (int i = 0; i < NF / 2; ++i) {
      const uint32_t t = bwa[i];
      bwa[i] = bwb[i];
      bwb[i] = t;
    }
  }
  if (ks < nks) {   // one or two steps left, in sets 0 and 1
    step_il<PAT, SPR>(acc, p.o0, b0, bwa, bwb, st0, st1, st2, p.o1, p.r1, p.w2, lane, [](auto) {}, lut);
    if (ks + 1 < nks) {
      __syncthreads();
      step_il<PAT, SPR>(acc, p.o1, b0, bwb, bwa, st1, st2, st0, p.o2, p.r2, p.w0, lane, [](auto) {}, lut);
    }
  }
}

// Epilogue.  2-byte outputs go through the wavefront's LDS region `epi` as
// whole row segments when the output allows 16-byte stores (every
// workgroup-uniform condition); otherwise each lane stores its own row, four
// consecutive columns per store.  The caller makes `epi` free.
template <typename OutT, int NF>
__device__ __forceinline__ void il_epilogue(const v16f (&acc)[NF], OutT* Y, int64_t ldy, int64_t row_lo,
                                            int64_t row_hi, int n0, int N, uint8_t* epi, int wave, int lane) {
  const int half = lane >> 5;
  if constexpr (sizeof(OutT) == 2) {
    if (((reinterpret_cast<uintptr_t>(Y) | (uintptr_t)(ldy * 2)) & 15u) == 0 && N % 8 == 0) {
      store_tile_lds<OutT, NF>(acc, Y, ldy, row_lo + wave * 32, row_hi, n0, N, epi, lane);
      return;
    }
  }
  const int64_t row = row_lo + wave * 32 + (lane & 31);
  if (row >= row_hi) return;
  OutT* yr = Y + row * ldy;
  const bool vec = ((reinterpret_cast<uintptr_t>(Y) | (uintptr_t)(ldy * (int64_t)sizeof(OutT))) &
                    (uintptr_t)(Vec4Out<OutT>::kAlign - 1)) == 0;
#pragma unroll
  for (int f = 0; f < NF; ++f) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col = n0 + f * 32 + 8 * g + 4 * half;
      if (vec && col + 3 < N) {
        Vec4Out<OutT>::put(yr + col, acc[f][4 * g], acc[f][4 * g + 1], acc[f][4 * g + 2], acc[f][4 * g + 3]);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e)
          if (col + e < N) store_out<OutT>(yr + col + e, acc[f][4 * g + e]);
      }
    }
  }
}

// This lane's activation row in a tile of rows [row_lo, row_hi): rows past
// the end are clamped (loads stay in bounds, stores are masked).
__device__ __forceinline__ int64_t il_row(const int32_t* row_index, int64_t row_lo, int64_t row_hi) {
  int64_t orow = row_lo + (threadIdx.x >> 6) * 32 + (threadIdx.x & 31);
  if (orow >= row_hi) orow = row_hi - 1;
  return row_index ? (int64_t)row_index[orow] : orow;
}

// One tile of the interleaved pipeline, alone: its LDS stages at lds, its
// epilogue staged over them once every wavefront is done with them.
template <int PAT, typename OutT, int NF>
__device__ __forceinline__ void tile_mx_il(const uint8_t* sp_codes, const uint8_t* sp_meta, const uint8_t* sp_scale,
                                           const uint8_t* dn_codes, const uint8_t* dn_scale, const int32_t* row_index,
                                           int64_t act_rows, int64_t row_lo, int64_t row_hi, const uint8_t* wc,
                                           const uint8_t* ws, int n0, int N, int K, OutT* Y, int64_t ldy,
                                           uint8_t* lds, const uint2* lut) {
  static_assert(NF == 8 || NF == 4, "full (256-column) or half tile");
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5;
  ARow a;
  a.r = il_row(row_index, row_lo, row_hi);
  a.R = act_rows;
  a.dn = dn_codes;
  a.spc = sp_codes;
  a.spm = sp_meta;
  a.dns = dn_scale;
  a.sps = sp_scale;
  v16f acc[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[f][r] = 0.0f;
  IlSets<NF> p;
  uint4 b0[NF];
  uint32_t bwa[NF / 2];
  il_issue<PAT, NF>(p, a, wc, ws, n0, N, K, half);
  il_start<PAT, NF>(p, wc, ws, n0, N, K, lds, b0, bwa, lane, half);
  il_main<PAT, NF>(acc, p, b0, bwa, a, wc, ws, n0, N, K, lds, lane, half, lut);
  __syncthreads();   // every wavefront is done with the weight stages
  il_epilogue<OutT, NF>(acc, Y, ldy, row_lo, row_hi, n0, N, lds + wave * kEpiWave, wave, lane);
}

// A tile of the persistent loops: output rows [row_lo, row_hi), this lane's
// activation row r, weight columns n0.. of the payload at wc / ws.
struct IlTile {
  int64_t row_lo, row_hi, r;
  const uint8_t *wc, *ws;
  int n0;
};

// Full tiles back to back, as handed out by next(IlTile&) until it returns
// false.  The next tile's first loads go out after the current tile's last
// step and before its output stores: the vector-memory counter completes in
// issue order, so loads issued behind the stores would first wait for the
// stores (64 KB per tile) to drain.  The epilogue therefore has its own LDS
// region `epi` (4 kEpiWave bytes) beside the three stages at `lds`.
template <int PAT, typename OutT, int SPR = 0, class Next>
__device__ __forceinline__ void tiles_mx_il(const uint8_t* sp_codes, const uint8_t* sp_meta, const uint8_t* sp_scale,
                                            const uint8_t* dn_codes, const uint8_t* dn_scale, int64_t act_rows, int N,
                                            int K, OutT* Y, int64_t ldy, uint8_t* lds, uint8_t* epi,
                                            const uint2* lut, Next next) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5;
  IlTile t;
  if (!next(t)) return;
  ARow a;
  a.r = t.r;
  a.R = act_rows;
  a.dn = dn_codes;
  a.spc = sp_codes;
  a.spm = sp_meta;
  a.dns = dn_scale;
  a.sps = sp_scale;
  IlSets<8> p;
  il_issue<PAT, 8>(p, a, t.wc, t.ws, t.n0, N, K, half);
  for (;;) {
    uint4 b0[8];
    uint32_t bwa[4];
    il_start<PAT, 8>(p, t.wc, t.ws, t.n0, N, K, lds, b0, bwa, lane, half);
    IlTile tn;
    const bool more = next(tn);   // the row-index load has the whole tile to arrive
    v16f acc[8];
#pragma unroll
    for (int f = 0; f < 8; ++f)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[f][r] = 0.0f;
    il_main<PAT, 8, SPR>(acc, p, b0, bwa, a, t.wc, t.ws, t.n0, N, K, lds, lane, half, lut);
    if (more) {
      a.r = tn.r;
      il_issue<PAT, 8>(p, a, tn.wc, tn.ws, tn.n0, N, K, half);
    }
    il_epilogue<OutT, 8>(acc, Y, ldy, t.row_lo, t.row_hi, t.n0, N, epi + wave * kEpiWave, wave, lane);
    if (!more) return;
    t = tn;
    __syncthreads();   // every wavefront is done with the stages before they are refilled
  }
}

// Tile order.  Workgroups are dispatched round-robin over the 8 XCDs
// (workgroup id mod 8), each with its own L2.  The ids are renumbered so that
// each XCD walks a contiguous range of tiles, ordered in blocks of 4 M-tiles
// x 8 N-tiles: the 32 workgroups an XCD runs at once then share 4 activation
// tiles and 8 weight tiles in its L2.  Other grid shapes keep row-major order.
__device__ __forceinline__ void tile_of(int id, int gx, int gy, int& mt, int& nt) {
  const int total = gx * gy;
  if ((gx & 7) == 0 && (gy & 3) == 0) {
    const int per = total >> 3;
    const int idp = (id & 7) * per + (id >> 3);
    const int blk = idp >> 5, in = idp & 31;
    const int bx = gx >> 3;
    mt = (blk / bx) * 4 + (in & 3);
    nt = (blk % bx) * 8 + (in >> 2);
  } else {
    mt = id / gx;
    nt = id - mt * gx;
  }
}

// The same order for any grid, for persistent loops: ids [0, 8 ceil(gx gy /
// 8)) map one to one onto tile numbers, XCD x (id mod 8) taking a contiguous
// range, walked in groups of 4 M-tiles, column by column (32 consecutive
// numbers are 4 M-tiles x 8 N-tiles, as in tile_of, which this equals when
// gx is a multiple of 8 and gy of 4).  False for the ids past the last tile.
__device__ __forceinline__ bool tile_at(int id, int gx, int gy, int& mt, int& nt) {
  const int total = gx * gy, per = (total + 7) >> 3;
  const int u = (id & 7) * per + (id >> 3);
  if (u >= total) return false;
  const int g = u / (4 * gx), first = 4 * g;
  const int gs = gy - first < 4 ? gy - first : 4;
  const int in = u - g * 4 * gx;
  mt = first + in % gs;
  nt = in / gs;
  return true;
}

// One tile per workgroup, for K not a multiple of 128 (the simpler pipeline
// of tile_mx, which handles a narrow last panel).
template <int NF, int PAT, bool SCALE_DW, typename OutT>
__global__ __launch_bounds__(256) void k_linear_mx(const uint8_t* sp_codes, const uint8_t* sp_meta,
                                                   const uint8_t* sp_scale, const uint8_t* dn_codes,
                                                   const uint8_t* dn_scale, int64_t M, const uint8_t* wc,
                                                   const uint8_t* ws, int N, int K, OutT* Y, int64_t ldy, int gx,
                                                   int gy) {
  constexpr int BN = 32 * NF;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * BN * kLdsStride + 2 * 64 * 2 * NF];
  uint8_t* lds_w = lds;
  uint8_t* lds_s = lds + 2 * BN * kLdsStride;
  int mt, nt;
  tile_of(blockIdx.x, gx, gy, mt, nt);
  const int n0 = nt * BN;
  const int64_t m0 = (int64_t)mt * kBM;
  const int64_t m1 = m0 + kBM < M ? m0 + kBM : M;
  tile_mx<NF, PAT, SCALE_DW, OutT>(sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, nullptr, M, m0, m1, wc, ws, n0, N,
                                   K, Y, ldy, lds_w, lds_s);
}

// Persistent dense kernel (K a multiple of 128): at most one workgroup per
// CU, walking the work units b, b + G, b + 2G, ... (G workgroups).  A tile's
// output stores then drain while the same CU starts its next tile instead of
// the whole grid waiting at the end of every round (3% on the Llama gate/up
// shape, 7 rounds).  With G a multiple of 8 every tile an XCD runs keeps the
// XCD of its number, so the tile_of blocks still share an L2.
//
// Units [0, full) are whole tiles.  When the last round would be at most
// half full (tiles = full + r, 0 < r <= G / 2), its r tiles run instead as
// 2 r half tiles of 128 columns, units [full, full + 2 r): every CU then
// runs a half tile instead of half of the CUs running a whole one (the
// Llama qkv shape: 384 tiles on 256 CUs).  Half tile u covers tile t(u),
// columns 128 h(u) on; with r a multiple of 8, t(u) keeps the XCD of u.
__device__ __forceinline__ void half_unit(int u, int full, int halves, int& t, int& h) {
  if ((halves & 15) == 0 && (full & 7) == 0) {
    t = full + ((u >> 4) << 3) + (u & 7);
    h = (u >> 3) & 1;
  } else {
    t = full + (u >> 1);
    h = u & 1;
  }
}

template <int PAT, typename OutT>
__global__ __launch_bounds__(256) void k_linear_mx_persist(const uint8_t* sp_codes, const uint8_t* sp_meta,
                                                           const uint8_t* sp_scale, const uint8_t* dn_codes,
                                                           const uint8_t* dn_scale, int64_t M, const uint8_t* wc,
                                                           const uint8_t* ws, int N, int K, OutT* Y, int64_t ldy,
                                                           int gx, int gy, int full, int halves) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[kPersistLds];
  __shared__ uint2 lut48[256];
  if (PAT == 48) {
    lut48_fill(lut48);
    __syncthreads();
  }
  int id = (int)blockIdx.x;
  tiles_mx_il<PAT, OutT>(sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, M, N, K, Y, ldy, lds,
                         lds + 3 * kStageBytes, lut48, [&](IlTile& t) {
                           if (id >= full) return false;
                           int mt, nt;
                           tile_of(id, gx, gy, mt, nt);
                           t.row_lo = (int64_t)mt * kBM;
                           t.row_hi = t.row_lo + kBM < M ? t.row_lo + kBM : M;
                           t.r = il_row(nullptr, t.row_lo, t.row_hi);
                           t.wc = wc;
                           t.ws = ws;
                           t.n0 = nt * 256;
                           id += (int)gridDim.x;
                           return true;
                         });
  for (; id < full + halves; id += (int)gridDim.x) {
    int t, h, mt, nt;
    half_unit(id - full, full, halves, t, h);
    tile_of(t, gx, gy, mt, nt);
    const int64_t m0 = (int64_t)mt * kBM;
    const int64_t m1 = m0 + kBM < M ? m0 + kBM : M;
    __syncthreads();   // the LDS stages are free before this tile's prologue
    tile_mx_il<PAT, OutT, 4>(sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, nullptr, M, m0, m1, wc, ws,
                             nt * 256 + 128 * h, N, K, Y, ldy, lds, lut48);
  }
}

// Grouped (MoE) form.  The grid is (column tiles) x (items); an item is a
// 128-row tile of one expert's slice [off[e], off[e+1]) of the output.  The
// tile-to-expert map is rebuilt on the device from expert_offsets (an
// exclusive scan of ceil(rows_e / 128)), so the host never reads the
// routing.  Items past the last tile exit before any barrier.
template <int NF, int PAT, bool SCALE_DW, typename OutT>
__global__ __launch_bounds__(256) void k_linear_mx_grouped(
    const uint8_t* sp_codes, const uint8_t* sp_meta, const uint8_t* sp_scale, const uint8_t* dn_codes,
    const uint8_t* dn_scale, const int32_t* row_index, int64_t act_rows, const int32_t* offs, int E,
    const uint8_t* wc, const uint8_t* ws, int N, int K, OutT* Y, int64_t ldy, int gx) {
  constexpr int BN = 32 * NF;
  constexpr int kOld = 2 * BN * kLdsStride + 2 * 64 * 2 * NF;
  __shared__ __attribute__((aligned(16))) uint8_t lds[kOld > kTileLds ? kOld : kTileLds];
  uint8_t* lds_w = lds;
  uint8_t* lds_s = lds + 2 * BN * kLdsStride;
  __shared__ int s_first[1025];
  const int tid = threadIdx.x;
  // tiles per expert, then an inclusive scan (Hillis-Steele) over <= 1024 experts
  for (int e = tid; e < E; e += 256) {
    const int rows = offs[e + 1] - offs[e];
    s_first[e + 1] = rows > 0 ? (rows + kBM - 1) / kBM : 0;
  }
  if (tid == 0) s_first[0] = 0;
  __syncthreads();
  for (int step = 1; step < E; step <<= 1) {
    int v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = tid + 256 * j + 1;
      v[j] = (e <= E && e - step >= 1) ? s_first[e - step] : 0;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = tid + 256 * j + 1;
      if (e <= E) s_first[e] += v[j];
    }
    __syncthreads();
  }
  // Workgroups go round-robin over the 8 XCDs; renumber so that each XCD
  // walks a contiguous range of (column tile, item) pairs in column-major
  // order: the few row tiles of one expert that share a weight tile then run
  // back to back on one XCD and reuse it from that XCD's L2.
  const int items = (int)gridDim.x / gx;
  const int total_wg = (int)gridDim.x;
  int idp = blockIdx.x;
  if ((total_wg & 7) == 0) idp = (blockIdx.x & 7) * (total_wg >> 3) + (blockIdx.x >> 3);
  const int xt = idp / items, item = idp - xt * items;
  if (item >= s_first[E]) return;   // uniform across the workgroup
  int lo = 0, hi = E;               // find e with s_first[e] <= item < s_first[e+1]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (s_first[mid] <= item) lo = mid; else hi = mid;
  }
  const int e = lo;
  const int64_t r0 = (int64_t)offs[e] + (int64_t)(item - s_first[e]) * kBM;
  const int64_t r_end = offs[e + 1];
  const int64_t r1 = r0 + kBM < r_end ? r0 + kBM : r_end;
  const int n0 = xt * BN;
  const uint8_t* wce = wc + (int64_t)e * N * (K / 2);
  const uint8_t* wse = ws + (int64_t)e * N * (K / 32);
  if constexpr (SCALE_DW && NF == 8)
  {
    __shared__ uint2 lut48[256];
    if (PAT == 48) {
      lut48_fill(lut48);
      __syncthreads();
    }
    tile_mx_il<PAT, OutT, 8>(sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, row_index, act_rows, r0, r1, wce, wse, n0,
                          N, K, Y, ldy, lds, lut48);
  }
  else
    tile_mx<NF, PAT, SCALE_DW, OutT>(sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, row_index, act_rows, r0, r1,
                                     wce, wse, n0, N, K, Y, ldy, lds_w, lds_s);
}

// Persistent grouped form (K a multiple of 128): at most one workgroup per
// CU walks the real (column tile, item) pairs -- their count comes from the
// same on-device scan -- so a CU starts its next tile without a new
// workgroup launch and the padding items of the launch-per-tile form cost
// nothing.  The order is XCD-contiguous and item-major: the column tiles of
// one row tile, and the few row tiles of one expert, run at the same time on
// one XCD and share its L2 (an item's gathered activation rows and the
// expert's weight tiles).  Measured on the Qwen3-30B-A3B experts (4096
// tokens, top-8): gate_up 190.7 -> 173.7 us, bit-identical; its 1902 units
// had fallen outside the earlier numbering, which required a multiple of 8,
// and were spread round-robin over the XCDs.  A last round at most half
// full runs as half tiles, as in the dense kernel (gate_up's 110 leftover
// units as 220 halves: 164.4 -> 162.8 us).  GATHER (a row map is given):
// full tiles take the spread load schedule of step5 (gate_up 165 -> 154 us,
// bit-identical; contiguous rows keep the burst, which is faster for them).
template <int PAT, typename OutT, bool GATHER = false>
__global__ __launch_bounds__(256) void k_linear_mx_grouped_persist(
    const uint8_t* sp_codes, const uint8_t* sp_meta, const uint8_t* sp_scale, const uint8_t* dn_codes,
    const uint8_t* dn_scale, const int32_t* row_index, int64_t act_rows, const int32_t* offs, int E,
    const uint8_t* wc, const uint8_t* ws, int N, int K, OutT* Y, int64_t ldy, int gx) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[kPersistLds];
  __shared__ int s_first[1025];
  __shared__ uint2 lut48[256];
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += 256) {
    const int rows = offs[e + 1] - offs[e];
    s_first[e + 1] = rows > 0 ? (rows + kBM - 1) / kBM : 0;
  }
  if (tid == 0) s_first[0] = 0;
  if (PAT == 48) lut48_fill(lut48);
  __syncthreads();
  for (int step = 1; step < E; step <<= 1) {
    int v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = tid + 256 * j + 1;
      v[j] = (e <= E && e - step >= 1) ? s_first[e - step] : 0;
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = tid + 256 * j + 1;
      if (e <= E) s_first[e] += v[j];
    }
    __syncthreads();
  }
  const int items = s_first[E];
  const int total = gx * items;
  // When the last round would be at most half full, its units run as twice
  // as many half tiles of 128 columns (as in k_linear_mx_persist).
  const int G = (int)gridDim.x, rem = total % G;
  const int halves = rem > 0 && 2 * rem <= G ? 2 * rem : 0;
  const int full = total - halves / 2;
  // unit u (item-major: item u / gx, column tile u mod gx) -> expert, rows
  const auto locate = [&](int u, int& e, int64_t& row_lo, int64_t& row_hi) {
    const int item = u / gx;
    int lo = 0, hi = E;   // e with s_first[e] <= item < s_first[e+1]
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (s_first[mid] <= item) lo = mid; else hi = mid;
    }
    e = lo;
    row_lo = (int64_t)offs[e] + (int64_t)(item - s_first[e]) * kBM;
    const int64_t r_end = offs[e + 1];
    row_hi = row_lo + kBM < r_end ? row_lo + kBM : r_end;
  };
  // XCD-contiguous numbering of the whole-tile units for any count: ids
  // [0, 8 per) map one to one onto units, XCD x (id mod 8) taking units
  // [x per, (x + 1) per); ids whose unit is past the last are skipped.
  const int per = (full + 7) >> 3;
  int id = (int)blockIdx.x;
  tiles_mx_il<PAT, OutT, GATHER ? 1 : 0>(sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, act_rows, N, K, Y, ldy, lds,
                         lds + 3 * kStageBytes, lut48, [&](IlTile& t) {
                           int u = full;
                           while (u >= full) {
                             if (id >= 8 * per) return false;
                             u = (id & 7) * per + (id >> 3);
                             id += G;
                           }
                           int e;
                           locate(u, e, t.row_lo, t.row_hi);
                           t.r = il_row(row_index, t.row_lo, t.row_hi);
                           t.wc = wc + (int64_t)e * N * (K / 2);
                           t.ws = ws + (int64_t)e * N * (K / 32);
                           t.n0 = (u % gx) * 256;
                           return true;
                         });
  if ((int)blockIdx.x < halves) {
    int u, h, e;
    half_unit((int)blockIdx.x, full, halves, u, h);
    int64_t row_lo, row_hi;
    locate(u, e, row_lo, row_hi);
    __syncthreads();   // the LDS stages are free before this tile's prologue
    tile_mx_il<PAT, OutT, 4>(sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, row_index, act_rows, row_lo, row_hi,
                             wc + (int64_t)e * N * (K / 2), ws + (int64_t)e * N * (K / 32), (u % gx) * 256 + 128 * h,
                             N, K, Y, ldy, lds, lut48);
  }
}

// ---------------------------------------------------------------------------
// Small-M (decode) MXFP4 GEMM
// ---------------------------------------------------------------------------
//
// With few activation rows the layer streams its weight from HBM and the
// prefill tile (128 x 256 outputs) leaves most CUs idle.  Here a workgroup
// owns 16 NB output columns and all M <= 16 MF rows, on the FP4 MFMA
// v_mfma_scale_f32_16x16x128_f8f6f4 (lane l holds row / column l % 16 and
// the 32 K values of block l / 16 of a 128-position panel; accumulator
// element r of lane l is row 4 (l / 16) + r, column l % 16).  Its KS
// wavefronts split K into KS ranges; each streams its weight slice straight
// from HBM into MFMA operands (1 KB loads per panel, coalesced by the
// panel-major layout) with a two-deep register prefetch, expands each
// activation block once for all NB column fragments, and the KS partial
// tiles are added in LDS in a fixed order.

typedef float v4f_t __attribute__((ext_vector_type(4)));

template <int MF, int NB>
struct SkinnyStage {
  uint4 w[NB];             // weight codes: column 16 n + l % 16, block l / 16
  uint32_t ws[NB];         // their E8M0 scales (bytes)
  uint4 dn[MF];            // residual codes of row 16 m + l % 16, block l / 16
  uint2 spc[MF];           // backbone codes and metadata of the same block
  uint32_t spm[MF];
  uint4 spd[MF];           // or (pattern 0) its dense backbone codes
  uint32_t sdn[MF], ssp[MF];
};

// PAT 0: spc is the dense backbone copy (16 bytes per block, the residual
// codes' layout) and spm is unused.
template <int MF, int NB, int PAT>
__device__ __forceinline__ void skinny_load(SkinnyStage<MF, NB>& st, const uint8_t* spc, const uint8_t* spm,
                                            const uint8_t* sps, const uint8_t* dnc, const uint8_t* dns, int64_t M,
                                            int64_t r0, const uint8_t* wc, const uint8_t* ws, int N, int n0, int ks,
                                            int lane) {
  const int j = lane >> 4;   // block within the panel
  const int64_t pn = (int64_t)ks * N, pm = (int64_t)ks * M;
#pragma unroll
  for (int n = 0; n < NB; ++n) {
    const int col = min(n0 + 16 * n + (lane & 15), N - 1);
    st.w[n] = *reinterpret_cast<const uint4*>(wc + (pn + col) * 64 + 16 * j);
    st.ws[n] = ws[(pn + col) * 4 + j];
  }
#pragma unroll
  for (int m = 0; m < MF; ++m) {
    int64_t row = r0 + 16 * m + (lane & 15);
    if (row >= M) row = M - 1;
    const int64_t V = (pm + row) * 4 + j;   // block-major index of (row, block)
    st.dn[m] = *reinterpret_cast<const uint4*>(dnc + V * 16);
    if (PAT == 0) {
      st.spd[m] = *reinterpret_cast<const uint4*>(spc + V * 16);
    } else {
      st.spc[m] = *reinterpret_cast<const uint2*>(spc + V * 8);
      st.spm[m] = *reinterpret_cast<const uint32_t*>(spm + V * 4);
    }
    st.sdn[m] = dns[V];
    st.ssp[m] = sps[V];
  }
}

// The weight is the MFMA's first operand: accumulator element r of lane l is
// then output column 4 (l / 16) + r of the fragment and activation row l % 16.
template <int MF, int NB, int PAT>
__device__ __forceinline__ void skinny_step(v4f_t (&acc)[MF][NB], const SkinnyStage<MF, NB>& st) {
#pragma unroll
  for (int m = 0; m < MF; ++m) {
    const v8i asp = as_operand(PAT == 0 ? st.spd[m] : expand_block<PAT>(st.spc[m], st.spm[m]));
    const v8i adn = as_operand(st.dn[m]);
#pragma unroll
    for (int n = 0; n < NB; ++n) {
      const v8i b = as_operand(st.w[n]);
      acc[m][n] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b, asp, acc[m][n], 4, 4, 0, (int)st.ws[n], 0,
                                                                  (int)st.ssp[m]);
      acc[m][n] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(b, adn, acc[m][n], 4, 4, 0, (int)st.ws[n], 0,
                                                                  (int)st.sdn[m]);
    }
  }
}

// Workgroup id -> (column group, row tile).  Workgroups are dispatched
// round-robin over the 8 XCDs; with several row tiles the ids are renumbered
// to give each XCD a contiguous range in which the row tiles of one column
// group follow each other, so the workgroups that read the same weight
// columns share an L2.
__device__ __forceinline__ void skinny_tile(int id, int ncg, int nrt, int& cg, int& rt) {
  if (nrt == 1) {
    cg = id;
    rt = 0;
    return;
  }
  const int total = ncg * nrt;
  const int idp = (total & 7) == 0 ? (id & 7) * (total >> 3) + (id >> 3) : id;
  cg = idp / nrt;
  rt = idp - cg * nrt;
}

template <int MF, int NB, int KS, int PAT, typename OutT>
__global__ __launch_bounds__(64 * KS) void k_linear_mx_skinny(const uint8_t* sp_codes, const uint8_t* sp_meta,
                                                              const uint8_t* sp_scale, const uint8_t* dn_codes,
                                                              const uint8_t* dn_scale, int64_t M, const uint8_t* wc,
                                                              const uint8_t* ws, int N, int K, OutT* Y, int64_t ldy,
                                                              int ncg, int nrt) {
  __shared__ float part[KS - 1][MF * NB][64][4];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  int cg, rt;
  skinny_tile(blockIdx.x, ncg, nrt, cg, rt);
  const int n0 = cg * 16 * NB;
  const int64_t r0 = (int64_t)rt * 16 * MF;
  const int nks = K / kBK;
  const int per = (nks + KS - 1) / KS;
  const int k0 = wave * per, k1 = min(nks, k0 + per);

  v4f_t acc[MF][NB];
#pragma unroll
  for (int m = 0; m < MF; ++m)
#pragma unroll
    for (int n = 0; n < NB; ++n) acc[m][n] = v4f_t{0.0f, 0.0f, 0.0f, 0.0f};

  SkinnyStage<MF, NB> s0, s1;
  if (k0 < k1)
    skinny_load<MF, NB, PAT>(s0, sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, M, r0, wc, ws, N, n0, k0, lane);
  if (k0 + 1 < k1)
    skinny_load<MF, NB, PAT>(s1, sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, M, r0, wc, ws, N, n0, k0 + 1, lane);
  int ks = k0;
  for (; ks + 1 < k1; ks += 2) {
    skinny_step<MF, NB, PAT>(acc, s0);
    if (ks + 2 < k1)
      skinny_load<MF, NB, PAT>(s0, sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, M, r0, wc, ws, N, n0, ks + 2, lane);
    skinny_step<MF, NB, PAT>(acc, s1);
    if (ks + 3 < k1)
      skinny_load<MF, NB, PAT>(s1, sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, M, r0, wc, ws, N, n0, ks + 3, lane);
  }
  if (ks < k1) skinny_step<MF, NB, PAT>(acc, s0);

  // partial tiles of wavefronts 1..KS-1 to LDS; wavefront 0 adds them in order
  if (wave > 0) {
#pragma unroll
    for (int m = 0; m < MF; ++m)
#pragma unroll
      for (int n = 0; n < NB; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) part[wave - 1][m * NB + n][lane][r] = acc[m][n][r];
  }
  __syncthreads();
  if (wave != 0) return;
  for (int w = 0; w < KS - 1; ++w)
#pragma unroll
    for (int m = 0; m < MF; ++m)
#pragma unroll
      for (int n = 0; n < NB; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[m][n][r] += part[w][m * NB + n][lane][r];
#pragma unroll
  for (int m = 0; m < MF; ++m) {
    const int64_t row = r0 + 16 * m + (lane & 15);
    if (row >= M) continue;
#pragma unroll
    for (int n = 0; n < NB; ++n)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int c = n0 + 16 * n + 4 * (lane >> 4) + r;
        if (c < N) store_out<OutT>(Y + row * ldy + c, acc[m][n][r]);
      }
  }
}

template <int MF, int NB, int KS, int PAT, typename OutT>
static hipError_t go_skinny(const uint8_t* spc, const uint8_t* spm, const uint8_t* sps, const uint8_t* dnc,
                            const uint8_t* dns, int64_t M, const uint8_t* wc, const uint8_t* ws, int N, int K,
                            void* Y, int64_t ldy, hipStream_t st) {
  const int ncg = (N + 16 * NB - 1) / (16 * NB);
  const int nrt = (int)((M + 16 * MF - 1) / (16 * MF));
  k_linear_mx_skinny<MF, NB, KS, PAT, OutT><<<dim3((unsigned)(ncg * nrt)), dim3(64 * KS), 0, st>>>(
      spc, spm, sps, dnc, dns, M, wc, ws, N, K, reinterpret_cast<OutT*>(Y), ldy, ncg, nrt);
  return hipGetLastError();
}

// K split: about 8192 weight streams in flight (wavefronts x column
// fragments per wavefront, for M > 16 wavefronts alone) to keep HBM busy,
// at least 4 panels per wavefront, at most `cap` wavefronts per workgroup.
static int skinny_split(int wgs, int K, int cap) {
  const int nks = K / kBK;
  int ks = 4;
  while (ks < cap && wgs * ks * 2 <= 8192 && nks >= 4 * ks * 2) ks *= 2;
  return ks;
}

// (row fragments, column fragments, K splits) by M: every activation block
// expansion feeds NB column fragments; the K split keeps enough wavefronts
// streaming the weight.  Above 16 rows the workgroups tile M by 32 or 64.
template <int PAT, typename OutT>
static hipError_t go_skinny_m(const uint8_t* spc, const uint8_t* spm, const uint8_t* sps, const uint8_t* dnc,
                              const uint8_t* dns, int64_t M, const uint8_t* wc, const uint8_t* ws, int N, int K,
                              void* Y, int64_t ldy, hipStream_t st) {
  if (M <= 16) {
    // Column fragments: as many as leave at least 192 workgroups (one
    // workgroup runs on one CU), since each activation block loaded and
    // expanded then feeds more weight columns.
    // Measured on the Llama decode shapes with the weight streamed from HBM
    // (µs, M = 1 / 16): qkv 6.3 / 7.6 -> 5.7 / 6.3 with 2 fragments, gate_up
    // 19.3 / 24.2 -> 16.3 / 17.3 with 4.  Sixteen wavefronts of 4 fragments
    // spill registers, hence the cap of 8.
    const int nb = (N + 63) / 64 >= 192 ? 4 : (N + 31) / 32 >= 192 ? 2 : 1;
    const int ks = skinny_split((N + 15) / 16, K, nb == 4 ? 8 : 16);
#define SHARQ_SKINNY1(NB_, KS_) \
  if (nb == NB_ && ks == KS_) return go_skinny<1, NB_, KS_, PAT, OutT>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
    SHARQ_SKINNY1(4, 4) SHARQ_SKINNY1(4, 8)
    SHARQ_SKINNY1(2, 4) SHARQ_SKINNY1(2, 8) SHARQ_SKINNY1(2, 16)
    SHARQ_SKINNY1(1, 4) SHARQ_SKINNY1(1, 8) SHARQ_SKINNY1(1, 16)
#undef SHARQ_SKINNY1
    return hipErrorInvalidValue;   // unreachable: (nb, ks) is one of the above
  }
  if (M <= 32) {
    // As at M <= 16, 4 column fragments when N leaves 192 workgroups of 64
    // columns (M = 32 gate_up from HBM: 32.1 -> 26.0 µs), else 2.
    const int ks = skinny_split((N + 15) / 16, K, 8);
    if ((N + 63) / 64 >= 192)
      return ks == 8 ? go_skinny<2, 4, 8, PAT, OutT>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st)
                     : go_skinny<2, 4, 4, PAT, OutT>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
    return ks == 8 ? go_skinny<2, 2, 8, PAT, OutT>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st)
                   : go_skinny<2, 2, 4, PAT, OutT>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
  }
  // Above 32 rows the workgroups tile M by 32 or 64.  Of the configurations
  // (row fragments, column fragments, K splits) below, those that leave at
  // least 192 workgroups (one workgroup runs on one CU; fewer leave CUs
  // idle), and of them the one whose wavefront count is nearest to 1024 in
  // ratio (ties to the first).  Measured on the Llama decode shapes with the
  // weight streamed from HBM (µs): M = 64 qkv 12.5 -> 11.8; M = 128 qkv
  // 23.6 -> 19.4, down 30.1 -> 28.5.
  struct Cfg { int mf, nb, ks; };
  constexpr Cfg cfgs[4] = {{4, 4, 4}, {2, 4, 4}, {2, 2, 4}, {2, 2, 8}};
  const auto wgs = [&](const Cfg& c) {
    return (int64_t)((N + 16 * c.nb - 1) / (16 * c.nb)) * ((M + 16 * c.mf - 1) / (16 * c.mf));
  };
  const auto dist = [](int64_t w) { return w >= 1024 ? (double)w / 1024.0 : 1024.0 / (double)w; };
  int best = -1;
  for (int pass = 0; pass < 2 && best < 0; ++pass)   // pass 1 only when no configuration has 192 workgroups
    for (int i = 0; i < 4; ++i)
      if ((pass == 1 || wgs(cfgs[i]) >= 192) &&
          (best < 0 || dist(wgs(cfgs[i]) * cfgs[i].ks) < dist(wgs(cfgs[best]) * cfgs[best].ks)))
        best = i;
  switch (best) {
    case 0: return go_skinny<4, 4, 4, PAT, OutT>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
    case 1: return go_skinny<2, 4, 4, PAT, OutT>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
    case 2: return go_skinny<2, 2, 4, PAT, OutT>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
    default: return go_skinny<2, 2, 8, PAT, OutT>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
  }
}

// The small-M kernel serves M <= 32, and M <= 256 while the main kernel
// would have fewer than 48 tiles of 128 x 256 (measured on the Llama decode
// shapes: at 48 tiles the two are even; at 112 the main kernel is faster,
// 32.5 against 41.1 µs for gate_up at M = 64 with the weight streamed from
// HBM, and twice as fast at M = 128).
static bool use_skinny(int64_t M, int N, int K) {
  if (K % kBK != 0) return false;
  if (M <= kSkinnyMaxM) return true;
  const int64_t tiles = ((M + kBM - 1) / kBM) * (int64_t)((N + 255) / 256);
  return M <= kSkinnyMaxRowTiled && tiles < 48;
}

template <int PAT>
static hipError_t go_skinny_dt(int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps,
                               const uint8_t* dnc, const uint8_t* dns, int64_t M, const uint8_t* wc,
                               const uint8_t* ws, int N, int K, void* Y, int64_t ldy, hipStream_t st) {
  if (ydt == 2) return go_skinny_m<PAT, float>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
  if (ydt == 1) return go_skinny_m<PAT, _Float16>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
  return go_skinny_m<PAT, uint16_t>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
}

// ---------------------------------------------------------------------------
// NVFP4 two-path GEMM
// ---------------------------------------------------------------------------
//
// NVFP4 block scales are E4M3 (not powers of two), which the block-scaled FP4
// MFMA cannot apply, and the products q * d of an E2M1 code and an E4M3 scale
// carry up to 6 significant bits -- exact in bf16 but not in FP8.  So both
// operands are dequantized to bf16 (q * d, exact) and multiplied on
// v_mfma_f32_32x32x16_bf16; the per-tensor scales S_x * S_w are applied once
// in the epilogue.  One K step is one 32-position block.  Activation
// fragments are dequantized in the registers of the wavefront that owns the
// rows; the weight tile is dequantized once per workgroup into LDS (bf16,
// 64 bytes per row, parts XOR-swizzled like the MXFP4 path).
//
// bf16 32x32x16 operand layout: lane l holds row l % 32 and K values
// 8 (l / 32) + 0..7; the accumulator layout is that of the FP4 MFMA.

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ int swz_nv(int row) { return ((row >> 1) ^ (row >> 3)) & 3; }

// Eight E2M1 codes (one dword, lower K in the lower nibble) times scale d ->
// eight exact bf16 values (4 dwords).  The fp32 products have at most 6
// significant bits, so dropping the low 16 bits is exact.
__device__ __forceinline__ uint4 dequant8_bf16(uint32_t codes, float d) {
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v2f v;
    switch (i) {
      case 0: v = fp4x2_decode<0>(codes); break;
      case 1: v = fp4x2_decode<1>(codes); break;
      case 2: v = fp4x2_decode<2>(codes); break;
      default: v = fp4x2_decode<3>(codes); break;
    }
    const float a = v.x * d, b = v.y * d;
    o[i] = __builtin_amdgcn_perm(__float_as_uint(b), __float_as_uint(a), 0x07060302u);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 q) {
  bf16x8 v;
  __builtin_memcpy(&v, &q, 16);
  return v;
}

struct NvA {         // one lane's activation data for one 32-position block
  uint4 dn;          // residual codes
  uint2 spc;         // compressed backbone codes
  uint32_t spm;      // backbone metadata
  uint32_t ssc;      // backbone E4M3 scale (byte 0)
  uint32_t dsc;      // residual E4M3 scales of the two 16-halves (bytes 0, 1)
};

struct NvW {         // one thread's weight row for one block
  uint4 codes;
  uint32_t sc;
};

__device__ __forceinline__ void load_nv_a(NvA& s, const ARow& a, int ks, int K) {
  const int p = ks >> 2, j = ks & 3, wp = min(128, K - 128 * p);
  const int64_t pr = (int64_t)p * a.R;
  s.dn = *reinterpret_cast<const uint4*>(a.dn + pr * 64 + a.r * (wp / 2) + 16 * j);
  s.spc = *reinterpret_cast<const uint2*>(a.spc + pr * 32 + a.r * (wp / 4) + 8 * j);
  s.spm = *reinterpret_cast<const uint32_t*>(a.spm + pr * 16 + a.r * (wp / 8) + 4 * j);
  s.ssc = a.sps[pr * 4 + a.r * (wp / 32) + j];
  s.dsc = *reinterpret_cast<const uint16_t*>(a.dns + pr * 8 + a.r * (wp / 16) + 2 * j);
}

template <int NF>
__device__ __forceinline__ void load_nv_w(NvW& w, const uint8_t* wc, const uint8_t* ws, int n0, int N, int K,
                                          int ks) {
  static_assert(NF == 8, "one weight row per thread");
  const int p = ks >> 2, j = ks & 3, wp = min(128, K - 128 * p);
  const int64_t pn = (int64_t)p * N;
  const int n = min(n0 + (int)threadIdx.x, N - 1);
  w.codes = *reinterpret_cast<const uint4*>(wc + pn * 64 + (int64_t)n * (wp / 2) + 16 * j);
  w.sc = ws[pn * 4 + (int64_t)n * (wp / 32) + j];
}

// Dequantize this thread's weight row (32 values) into the LDS tile as bf16.
__device__ __forceinline__ void store_nv_w(const NvW& w, uint8_t* lds) {
  const int row = threadIdx.x;
  const float d = e4m3_value(w.sc);
  const uint32_t c[4] = {w.codes.x, w.codes.y, w.codes.z, w.codes.w};
#pragma unroll
  for (int q = 0; q < 4; ++q)
    *reinterpret_cast<uint4*>(lds + row * 64 + 16 * (q ^ swz_nv(row))) = dequant8_bf16(c[q], d);
}

template <int PAT, int NF>
__device__ __forceinline__ void step_nv(v16f (&acc)[NF], const NvA& a, const uint8_t* lw, int lane) {
  const int half = lane >> 5, col = lane & 31;
  const uint4 sp = expand_block<PAT>(a.spc, a.spm);
  const float dsp = e4m3_value(a.ssc & 0xFFu);
  const float d0 = e4m3_value(a.dsc & 0xFFu), d1 = e4m3_value((a.dsc >> 8) & 0xFFu);
  const uint32_t spw[4] = {sp.x, sp.y, sp.z, sp.w};
  const uint32_t dnw[4] = {a.dn.x, a.dn.y, a.dn.z, a.dn.w};
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    // K values 8 half + 16 t + 0..7: dword (half + 2 t) of the block; the
    // residual's 16-half is t
    const bf16x8 asp = as_bf16x8(dequant8_bf16(spw[half + 2 * t], dsp));
    const bf16x8 adn = as_bf16x8(dequant8_bf16(dnw[half + 2 * t], t ? d1 : d0));
    bf16x8 b[NF];
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const int row = f * 32 + col;
      b[f] = as_bf16x8(*reinterpret_cast<const uint4*>(lw + row * 64 + 16 * ((half + 2 * t) ^ swz_nv(row))));
    }
#pragma unroll
    for (int f = 0; f < NF; ++f) acc[f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(asp, b[f], acc[f], 0, 0, 0);
#pragma unroll
    for (int f = 0; f < NF; ++f) acc[f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(adn, b[f], acc[f], 0, 0, 0);
  }
}

template <int NF, int PAT, typename OutT>
__global__ __launch_bounds__(256) void k_linear_nv(const uint8_t* sp_codes, const uint8_t* sp_meta,
                                                   const uint8_t* sp_scale, const uint8_t* dn_codes,
                                                   const uint8_t* dn_scale, const float* ts_x, int64_t M,
                                                   const uint8_t* wc, const uint8_t* ws, const float* ts_w, int N,
                                                   int K, OutT* Y, int64_t ldy, int gx, int gy) {
  constexpr int BN = 32 * NF;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * BN * 64];
  int mt, nt;
  tile_of(blockIdx.x, gx, gy, mt, nt);
  const int n0 = nt * BN;
  const int64_t row_lo = (int64_t)mt * kBM;
  const int64_t row_hi = row_lo + kBM < M ? row_lo + kBM : M;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5;
  const int nks = K / 32;

  int64_t orow = row_lo + wave * 32 + (lane & 31);
  if (orow >= row_hi) orow = row_hi - 1;
  ARow a;
  a.r = orow;
  a.R = M;
  a.dn = dn_codes;
  a.spc = sp_codes;
  a.spm = sp_meta;
  a.dns = dn_scale;
  a.sps = sp_scale;

  v16f acc[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[f][r] = 0.0f;

  NvA a0, a1;
  NvW wn;
  const int last = nks - 1;
  load_nv_w<NF>(wn, wc, ws, n0, N, K, 0);
  load_nv_a(a0, a, 0, K);
  store_nv_w(wn, lds);
  load_nv_w<NF>(wn, wc, ws, n0, N, K, min(1, last));
  load_nv_a(a1, a, min(1, last), K);
  int ks = 0;
  for (; ks + 1 < nks; ks += 2) {
    __syncthreads();
    step_nv<PAT, NF>(acc, a0, lds, lane);
    store_nv_w(wn, lds + BN * 64);
    load_nv_w<NF>(wn, wc, ws, n0, N, K, min(ks + 2, last));
    load_nv_a(a0, a, min(ks + 2, last), K);
    __syncthreads();
    step_nv<PAT, NF>(acc, a1, lds + BN * 64, lane);
    store_nv_w(wn, lds);
    load_nv_w<NF>(wn, wc, ws, n0, N, K, min(ks + 3, last));
    load_nv_a(a1, a, min(ks + 3, last), K);
  }
  if (ks < nks) {
    __syncthreads();
    step_nv<PAT, NF>(acc, a0, lds, lane);
  }

  const float scale = *ts_x * *ts_w;
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int col = n0 + f * 32 + (lane & 31);
    if (col >= N) continue;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int64_t row = row_lo + wave * 32 + 8 * (r / 4) + 4 * half + (r % 4);
      if (row < row_hi) store_out<OutT>(Y + row * ldy + col, acc[f][r] * scale);
    }
  }
}

// ---------------------------------------------------------------------------
// Interleaved NVFP4 main loop (K a multiple of 128)
// ---------------------------------------------------------------------------
//
// The same slot schedule as the MXFP4 loop, on v_mfma_f32_32x32x16_f16 with
// the weight as first operand (each lane then owns an output row).  One K
// step is one 32-position block: two 16-position MFMA sub-steps t, where lane
// half h supplies positions 16 h + 8 t + 0..7 -- so a lane needs only its
// half of each block (one residual scale, 8 bytes of residual codes, half the
// backbone).  Between the step's 32 MFMAs run the weight reads of sub-step 1,
// the fp16 dequantization of the next step's activations, the dequantization
// and LDS store of the weight two steps ahead (three LDS stages) and the
// reads of the next step's first weight operands.

struct NvRaw {          // this lane's raw activation data of one step
  uint2 dn;             // residual codes of positions 16 h + 0..15
  uint32_t spc;         // compressed backbone codes of the same 16 positions;
                        // from the dense backbone copy (PAT 0): their first 8 codes
  uint32_t spm;         // their metadata (low 16 bits); PAT 0: the last 8 codes
  uint32_t ssc, dsc;    // backbone and residual E4M3 scales (bytes)
};

struct NvOps {          // MFMA-ready fp16 operands of one step
  uint4 sp[2], dn[2];
};

struct NvWRaw {         // one weight row of one step
  uint4 codes;
  uint32_t sc;
};

constexpr int kNvStage = 256 * 64;   // fp16 weight tile of one step: 256 rows x 32 positions

// Pieces of the exact dequantization q * d in fp16: codes byte SEL (two
// E2M1 values, lower position in the low nibble) -> one packed fp16 pair.
// Every such product is exact in fp16: q has at most 2 significant bits and
// |q| <= 6, an E4M3 scale d has at most 4 and lies in [2^-9, 448], so q d has
// at most 6 significant bits and lies in [2^-10, 2688], inside fp16's normal
// range.  The FP4 pair is decoded to fp16 and scaled by one packed fp16
// multiply (two values per instruction), half the work of decoding to fp32,
// scaling and packing to bf16.
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ f16x8 as_f16x8(uint4 q) {
  f16x8 v;
  __builtin_memcpy(&v, &q, 16);
  return v;
}

// an E4M3 scale as an fp16 pair (exact)
__device__ __forceinline__ f16x2 nv_scale2(uint32_t code) {
  const _Float16 h = (_Float16)e4m3_value(code);
  return f16x2{h, h};
}

template <int SEL>
__device__ __forceinline__ uint32_t f16_pair(uint32_t codes, f16x2 d) {
  const f16x2 v = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(codes, 1.0f, SEL);
  return __builtin_bit_cast(uint32_t, v * d);
}

// PAT 0: a.spc is the dense backbone copy (16 bytes per block, block-major).
template <int PAT>
__device__ __forceinline__ void nv_load_a(NvRaw& s, const ARow& a, int ks, int half) {
  const int64_t V = ((int64_t)(ks >> 2) * a.R + a.r) * 4 + (ks & 3);   // block-major index
  s.dn = *reinterpret_cast<const uint2*>(a.dn + V * 16 + 8 * half);
  if (PAT == 0) {
    const uint2 c = *reinterpret_cast<const uint2*>(a.spc + V * 16 + 8 * half);
    s.spc = c.x;
    s.spm = c.y;
  } else {
    s.spc = *reinterpret_cast<const uint32_t*>(a.spc + V * 8 + 4 * half);
    s.spm = (uint32_t)*reinterpret_cast<const uint16_t*>(a.spm + V * 4 + 2 * half);
  }
  s.ssc = a.sps[V];
  s.dsc = a.dns[V * 2 + half];
}

// Dense backbone codes D (0: positions 16 h + 0..7, 1: + 8..15) of a step:
// read as they are from the dense copy, or expanded from the compressed form.
template <int PAT, int D>
__device__ __forceinline__ uint32_t nv_backbone_dw(const NvRaw& r) {
  if (PAT == 0) return D == 0 ? r.spc : r.spm;
  return expand_dw<PAT, D>(make_uint2(r.spc, 0u), r.spm);
}

__device__ __forceinline__ void nv_load_w(NvWRaw& w, const uint8_t* wc, const uint8_t* ws, int n0, int N, int ks) {
  const int n = min(n0 + (int)threadIdx.x, N - 1);
  const int64_t V = ((int64_t)(ks >> 2) * N + n) * 4 + (ks & 3);
  w.codes = *reinterpret_cast<const uint4*>(wc + V * 16);
  w.sc = ws[V];
}

template <int SUB, int F0, int F1>
__device__ __forceinline__ void nv_read_b(uint4 (&b)[8], const uint8_t* lw, int lane) {
  const int half = lane >> 5, col = lane & 31;
#pragma unroll
  for (int f = F0; f < F1; ++f) {
    const int row = f * 32 + col;
    b[f] = *reinterpret_cast<const uint4*>(lw + row * 64 + 16 * ((2 * half + SUB) ^ swz_nv(row)));
  }
}

template <int SUB, int F>
__device__ __forceinline__ void nv_mma(v16f (&acc)[8], const uint4& a, const uint4 (&b)[8]) {
  acc[F] = __builtin_amdgcn_mfma_f32_32x32x16_f16(as_f16x8(b[F]), as_f16x8(a), acc[F], 0, 0, 0);
}

template <int PAT, class Issue>
__device__ __forceinline__ void nv_step(v16f (&acc)[8], const NvOps& ops, uint4 (&b0)[8], const uint8_t* cur,
                                        const uint8_t* nxt, uint8_t* wr, NvOps& opsn, const NvRaw& raw,
                                        const NvWRaw& wst, int lane, Issue issue) {
  const int tid = threadIdx.x;
  uint4 b1[8];
  issue();
  SHARQ_FENCE();
  // next step's activations: backbone expanded to 16 codes, then dequantized
  // (their scales decoded behind the first two MFMAs)
  f16x2 dsp, ddn;
  uint32_t e0 = 0u, e1 = 0u;
  // ---- sub-step 0, backbone
  nv_mma<0, 0>(acc, ops.sp[0], b0); nv_read_b<1, 0, 1>(b1, cur, lane); dsp = nv_scale2(raw.ssc); SHARQ_FENCE();
  nv_mma<0, 1>(acc, ops.sp[0], b0); nv_read_b<1, 1, 2>(b1, cur, lane); ddn = nv_scale2(raw.dsc);
  e0 = nv_backbone_dw<PAT, 0>(raw); SHARQ_FENCE();
  nv_mma<0, 2>(acc, ops.sp[0], b0); nv_read_b<1, 2, 3>(b1, cur, lane); SHARQ_FENCE();
  nv_mma<0, 3>(acc, ops.sp[0], b0); nv_read_b<1, 3, 4>(b1, cur, lane); e1 = nv_backbone_dw<PAT, 1>(raw); SHARQ_FENCE();
  nv_mma<0, 4>(acc, ops.sp[0], b0); nv_read_b<1, 4, 5>(b1, cur, lane);
  opsn.sp[0].x = f16_pair<0>(e0, dsp); opsn.sp[0].y = f16_pair<1>(e0, dsp); SHARQ_FENCE();
  nv_mma<0, 5>(acc, ops.sp[0], b0); nv_read_b<1, 5, 6>(b1, cur, lane);
  opsn.sp[0].z = f16_pair<2>(e0, dsp); opsn.sp[0].w = f16_pair<3>(e0, dsp); SHARQ_FENCE();
  nv_mma<0, 6>(acc, ops.sp[0], b0); nv_read_b<1, 6, 7>(b1, cur, lane);
  opsn.sp[1].x = f16_pair<0>(e1, dsp); opsn.sp[1].y = f16_pair<1>(e1, dsp); SHARQ_FENCE();
  nv_mma<0, 7>(acc, ops.sp[0], b0); nv_read_b<1, 7, 8>(b1, cur, lane);
  opsn.sp[1].z = f16_pair<2>(e1, dsp); opsn.sp[1].w = f16_pair<3>(e1, dsp); SHARQ_FENCE();
  // ---- sub-step 0, residual
  nv_mma<0, 0>(acc, ops.dn[0], b0);
  opsn.dn[0].x = f16_pair<0>(raw.dn.x, ddn); opsn.dn[0].y = f16_pair<1>(raw.dn.x, ddn); SHARQ_FENCE();
  nv_mma<0, 1>(acc, ops.dn[0], b0);
  opsn.dn[0].z = f16_pair<2>(raw.dn.x, ddn); opsn.dn[0].w = f16_pair<3>(raw.dn.x, ddn); SHARQ_FENCE();
  nv_mma<0, 2>(acc, ops.dn[0], b0);
  opsn.dn[1].x = f16_pair<0>(raw.dn.y, ddn); opsn.dn[1].y = f16_pair<1>(raw.dn.y, ddn); SHARQ_FENCE();
  nv_mma<0, 3>(acc, ops.dn[0], b0);
  opsn.dn[1].z = f16_pair<2>(raw.dn.y, ddn); opsn.dn[1].w = f16_pair<3>(raw.dn.y, ddn); SHARQ_FENCE();
  // the weight row two steps ahead: dequantized into the other stage, each
  // 16-byte part over two slots (4 values per slot)
  const f16x2 dw = nv_scale2(wst.sc);
  const int wrow = tid;
  uint32_t wx, wy;
  nv_mma<0, 4>(acc, ops.dn[0], b0);
  wx = f16_pair<0>(wst.codes.x, dw); wy = f16_pair<1>(wst.codes.x, dw); SHARQ_FENCE();
  nv_mma<0, 5>(acc, ops.dn[0], b0);
  *reinterpret_cast<uint4*>(wr + wrow * 64 + 16 * (0 ^ swz_nv(wrow))) =
      make_uint4(wx, wy, f16_pair<2>(wst.codes.x, dw), f16_pair<3>(wst.codes.x, dw));
  SHARQ_FENCE();
  nv_mma<0, 6>(acc, ops.dn[0], b0);
  wx = f16_pair<0>(wst.codes.y, dw); wy = f16_pair<1>(wst.codes.y, dw); SHARQ_FENCE();
  nv_mma<0, 7>(acc, ops.dn[0], b0);
  *reinterpret_cast<uint4*>(wr + wrow * 64 + 16 * (1 ^ swz_nv(wrow))) =
      make_uint4(wx, wy, f16_pair<2>(wst.codes.y, dw), f16_pair<3>(wst.codes.y, dw));
  SHARQ_FENCE();
  // ---- sub-step 1, backbone
  nv_mma<1, 0>(acc, ops.sp[1], b1);
  wx = f16_pair<0>(wst.codes.z, dw); wy = f16_pair<1>(wst.codes.z, dw); SHARQ_FENCE();
  nv_mma<1, 1>(acc, ops.sp[1], b1);
  *reinterpret_cast<uint4*>(wr + wrow * 64 + 16 * (2 ^ swz_nv(wrow))) =
      make_uint4(wx, wy, f16_pair<2>(wst.codes.z, dw), f16_pair<3>(wst.codes.z, dw));
  SHARQ_FENCE();
  nv_mma<1, 2>(acc, ops.sp[1], b1);
  wx = f16_pair<0>(wst.codes.w, dw); wy = f16_pair<1>(wst.codes.w, dw); SHARQ_FENCE();
  nv_mma<1, 3>(acc, ops.sp[1], b1);
  *reinterpret_cast<uint4*>(wr + wrow * 64 + 16 * (3 ^ swz_nv(wrow))) =
      make_uint4(wx, wy, f16_pair<2>(wst.codes.w, dw), f16_pair<3>(wst.codes.w, dw));
  SHARQ_FENCE();
  nv_mma<1, 4>(acc, ops.sp[1], b1); SHARQ_FENCE();
  nv_mma<1, 5>(acc, ops.sp[1], b1); SHARQ_FENCE();
  nv_mma<1, 6>(acc, ops.sp[1], b1); SHARQ_FENCE();
  nv_mma<1, 7>(acc, ops.sp[1], b1); SHARQ_FENCE();
  // ---- sub-step 1, residual; the next step's first weight operands
  nv_mma<1, 0>(acc, ops.dn[1], b1); nv_read_b<0, 0, 1>(b0, nxt, lane); SHARQ_FENCE();
  nv_mma<1, 1>(acc, ops.dn[1], b1); nv_read_b<0, 1, 2>(b0, nxt, lane); SHARQ_FENCE();
  nv_mma<1, 2>(acc, ops.dn[1], b1); nv_read_b<0, 2, 3>(b0, nxt, lane); SHARQ_FENCE();
  nv_mma<1, 3>(acc, ops.dn[1], b1); nv_read_b<0, 3, 4>(b0, nxt, lane); SHARQ_FENCE();
  nv_mma<1, 4>(acc, ops.dn[1], b1); nv_read_b<0, 4, 5>(b0, nxt, lane); SHARQ_FENCE();
  nv_mma<1, 5>(acc, ops.dn[1], b1); nv_read_b<0, 5, 6>(b0, nxt, lane); SHARQ_FENCE();
  nv_mma<1, 6>(acc, ops.dn[1], b1); nv_read_b<0, 6, 7>(b0, nxt, lane); SHARQ_FENCE();
  nv_mma<1, 7>(acc, ops.dn[1], b1); nv_read_b<0, 7, 8>(b0, nxt, lane); SHARQ_FENCE();
}

template <int PAT>
__device__ __forceinline__ void nv_ops_from_raw(NvOps& o, const NvRaw& r) {
  const f16x2 dsp = nv_scale2(r.ssc), ddn = nv_scale2(r.dsc);
  const uint32_t e0 = nv_backbone_dw<PAT, 0>(r), e1 = nv_backbone_dw<PAT, 1>(r);
  o.sp[0] = make_uint4(f16_pair<0>(e0, dsp), f16_pair<1>(e0, dsp), f16_pair<2>(e0, dsp), f16_pair<3>(e0, dsp));
  o.sp[1] = make_uint4(f16_pair<0>(e1, dsp), f16_pair<1>(e1, dsp), f16_pair<2>(e1, dsp), f16_pair<3>(e1, dsp));
  o.dn[0] = make_uint4(f16_pair<0>(r.dn.x, ddn), f16_pair<1>(r.dn.x, ddn), f16_pair<2>(r.dn.x, ddn),
                       f16_pair<3>(r.dn.x, ddn));
  o.dn[1] = make_uint4(f16_pair<0>(r.dn.y, ddn), f16_pair<1>(r.dn.y, ddn), f16_pair<2>(r.dn.y, ddn),
                       f16_pair<3>(r.dn.y, ddn));
}

__device__ __forceinline__ void nv_store_w(const NvWRaw& w, uint8_t* stage) {
  const int row = threadIdx.x;
  const f16x2 d = nv_scale2(w.sc);
  const uint32_t c[4] = {w.codes.x, w.codes.y, w.codes.z, w.codes.w};
#pragma unroll
  for (int q = 0; q < 4; ++q)
    *reinterpret_cast<uint4*>(stage + row * 64 + 16 * (q ^ swz_nv(row))) =
        make_uint4(f16_pair<0>(c[q], d), f16_pair<1>(c[q], d), f16_pair<2>(c[q], d), f16_pair<3>(c[q], d));
}

template <int PAT, typename OutT>
__device__ __forceinline__ void tile_nv_il(const uint8_t* sp_codes, const uint8_t* sp_meta,
                                           const uint8_t* sp_scale, const uint8_t* dn_codes,
                                           const uint8_t* dn_scale, const float* ts_x, int64_t M,
                                           const uint8_t* wc, const uint8_t* ws, const float* ts_w, int N, int K,
                                           OutT* Y, int64_t ldy, int mt, int nt, uint8_t* lds) {
  constexpr int NF = 8;
  const int n0 = nt * 256;
  const int64_t row_lo = (int64_t)mt * kBM;
  const int64_t row_hi = row_lo + kBM < M ? row_lo + kBM : M;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5;
  const int nks = K / 32;   // one step per 32-position block

  int64_t orow = row_lo + wave * 32 + (lane & 31);
  if (orow >= row_hi) orow = row_hi - 1;   // clamp: loads stay in bounds, stores are masked
  ARow a;
  a.r = orow;
  a.R = M;
  a.dn = dn_codes;
  a.spc = sp_codes;
  a.spm = sp_meta;
  a.dns = dn_scale;
  a.sps = sp_scale;

  v16f acc[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[f][r] = 0.0f;

  // invariant at step k (sets by k mod 2, stages by k mod 3): stages k, k+1
  // hold W(k), W(k+1); b0 = step k's first operands; o[k] ready;
  // r[k+1] = raw A(k+1); w[k] = raw W(k+2)
  const int last = nks - 1;
  const auto cl = [&](int k) { return k < last ? k : last; };
  NvRaw r0, r1;
  NvWRaw w0, w1;
  NvOps o0, o1;
  uint4 b0[8];
  uint8_t* st0 = lds;
  uint8_t* st1 = lds + kNvStage;
  uint8_t* st2 = lds + 2 * kNvStage;
  nv_load_w(w0, wc, ws, n0, N, 0);
  nv_load_w(w1, wc, ws, n0, N, cl(1));
  nv_load_a<PAT>(r0, a, 0, half);
  nv_load_a<PAT>(r1, a, cl(1), half);
  nv_store_w(w0, st0);
  nv_store_w(w1, st1);
  nv_ops_from_raw<PAT>(o0, r0);
  nv_load_w(w0, wc, ws, n0, N, cl(2));
  __syncthreads();
  nv_read_b<0, 0, 8>(b0, st0, lane);

  int ks = 0;
  for (; ks + 1 < nks; ks += 2) {
    nv_step<PAT>(acc, o0, b0, st0, st1, st2, o1, r1, w0, lane, [&] {
      nv_load_w(w1, wc, ws, n0, N, cl(ks + 3));
      nv_load_a<PAT>(r0, a, cl(ks + 2), half);
    });
    __syncthreads();
    nv_step<PAT>(acc, o1, b0, st1, st2, st0, o0, r0, w1, lane, [&] {
      nv_load_w(w0, wc, ws, n0, N, cl(ks + 4));
      nv_load_a<PAT>(r1, a, cl(ks + 3), half);
    });
    __syncthreads();
    uint8_t* t = st0;   // rotate the stages by two
    st0 = st2;
    st2 = st1;
    st1 = t;
  }
  if (ks < nks) nv_step<PAT>(acc, o0, b0, st0, st1, st2, o1, r1, w0, lane, [] {});

  const float scale = *ts_x * *ts_w;
  const int64_t row = row_lo + wave * 32 + (lane & 31);
  if (row >= row_hi) return;
  OutT* yr = Y + row * ldy;
  const bool vec = ((reinterpret_cast<uintptr_t>(Y) | (uintptr_t)(ldy * (int64_t)sizeof(OutT))) &
                    (uintptr_t)(Vec4Out<OutT>::kAlign - 1)) == 0;
#pragma unroll
  for (int f = 0; f < NF; ++f) {
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int col = n0 + f * 32 + 8 * g + 4 * half;
      const float v0 = acc[f][4 * g] * scale, v1 = acc[f][4 * g + 1] * scale;
      const float v2 = acc[f][4 * g + 2] * scale, v3 = acc[f][4 * g + 3] * scale;
      if (vec && col + 3 < N) {
        Vec4Out<OutT>::put(yr + col, v0, v1, v2, v3);
      } else {
        if (col < N) store_out<OutT>(yr + col, v0);
        if (col + 1 < N) store_out<OutT>(yr + col + 1, v1);
        if (col + 2 < N) store_out<OutT>(yr + col + 2, v2);
        if (col + 3 < N) store_out<OutT>(yr + col + 3, v3);
      }
    }
  }
}

static int device_cus();   // compute units of the current device (host launchers below)

// Persistent: at most one workgroup per CU walks the tiles b, b + G, ... in
// the XCD-aware order of tile_at (any grid: the Qwen2.5-7B shapes have 148
// and 14 column tiles; measured neutral there, where the dequantization and
// MFMA work bound the kernel).
template <int PAT, typename OutT>
__global__ __launch_bounds__(256) void k_linear_nv_il(const uint8_t* sp_codes, const uint8_t* sp_meta,
                                                      const uint8_t* sp_scale, const uint8_t* dn_codes,
                                                      const uint8_t* dn_scale, const float* ts_x, int64_t M,
                                                      const uint8_t* wc, const uint8_t* ws, const float* ts_w, int N,
                                                      int K, OutT* Y, int64_t ldy, int gx, int gy) {
  __shared__ __attribute__((aligned(16))) uint8_t lds[3 * kNvStage];
  const int ids = 8 * ((gx * gy + 7) >> 3);
  for (int id = (int)blockIdx.x; id < ids; id += (int)gridDim.x) {
    int mt, nt;
    if (!tile_at(id, gx, gy, mt, nt)) continue;   // uniform across the workgroup
    tile_nv_il<PAT, OutT>(sp_codes, sp_meta, sp_scale, dn_codes, dn_scale, ts_x, M, wc, ws, ts_w, N, K, Y, ldy, mt, nt,
                          lds);
    __syncthreads();   // the LDS stages are free before the next tile's prologue
  }
}

template <int PAT, typename OutT>
static hipError_t go_nv(const uint8_t* spc, const uint8_t* spm, const uint8_t* sps, const uint8_t* dnc,
                        const uint8_t* dns, const float* tsx, int64_t M, const uint8_t* wc, const uint8_t* ws,
                        const float* tsw, int N, int K, void* Y, int64_t ldy, hipStream_t st) {
  constexpr int NF = 8;
  const int gx = (N + 32 * NF - 1) / (32 * NF), gy = (int)((M + kBM - 1) / kBM);
  if (K % kBK == 0) {
    const int tiles = gx * gy, cus = device_cus();
    k_linear_nv_il<PAT, OutT><<<dim3((unsigned)(tiles < cus ? tiles : cus)), dim3(256), 0, st>>>(
        spc, spm, sps, dnc, dns, tsx, M, wc, ws, tsw, N, K, reinterpret_cast<OutT*>(Y), ldy, gx, gy);
    return hipGetLastError();
  }
  if constexpr (PAT == 0) {
    return hipErrorInvalidValue;   // the dense backbone copy needs K a multiple of 128
  } else {
    k_linear_nv<NF, PAT, OutT><<<dim3((unsigned)(gx * gy)), dim3(256), 0, st>>>(
        spc, spm, sps, dnc, dns, tsx, M, wc, ws, tsw, N, K, reinterpret_cast<OutT*>(Y), ldy, gx, gy);
    return hipGetLastError();
  }
}

template <int PAT>
static hipError_t go_nv_dt(int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps, const uint8_t* dnc,
                           const uint8_t* dns, const float* tsx, int64_t M, const uint8_t* wc, const uint8_t* ws,
                           const float* tsw, int N, int K, void* Y, int64_t ldy, hipStream_t st) {
  if (ydt == 2) return go_nv<PAT, float>(spc, spm, sps, dnc, dns, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
  if (ydt == 1) return go_nv<PAT, _Float16>(spc, spm, sps, dnc, dns, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
  return go_nv<PAT, uint16_t>(spc, spm, sps, dnc, dns, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
}

hipError_t launch_linear_nv(int pat, int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps,
                            const uint8_t* dnc, const uint8_t* dns, const float* tsx, int64_t M, const uint8_t* wc,
                            const uint8_t* ws, const float* tsw, int N, int K, void* Y, int64_t ldy,
                            const uint8_t* spd, hipStream_t st) {
  if (spd && K % kBK == 0) return go_nv_dt<0>(ydt, spd, nullptr, sps, dnc, dns, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
  if (spc == nullptr) return hipErrorInvalidValue;   // rejected by the C ABI (K not a multiple of 128)
  return pat == 24 ? go_nv_dt<24>(ydt, spc, spm, sps, dnc, dns, tsx, M, wc, ws, tsw, N, K, Y, ldy, st)
                   : go_nv_dt<48>(ydt, spc, spm, sps, dnc, dns, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
}

// ---------------------------------------------------------------------------
// Path combinations (Sec. 4.4, table "ablation-combination"): the sum of up
// to two paths, each sparse (compressed codes + metadata, expanded in
// registers; scale per 32 logical positions) or dense (plain codes), into one
// accumulator.  Path 1 reads the sp_* buffers, path 2 the dn_* buffers.  A
// slot kind is 0 (absent), kSlotDense, or the sparse metadata layout (24 for
// 2:4, 48 for 4:8).  Generic kernels -- one tile per workgroup, double-
// buffered weight stages, any K a multiple of 32 -- since the combinations
// other than SharQ's exist for ablation.
// ---------------------------------------------------------------------------

constexpr int kSlotDense = 1;

struct SlotBuf {
  const uint8_t *c, *m, *s;   // codes, metadata (sparse only), scales
};

// One slot's data of one MXFP4 K step for this lane: per sub-step the codes
// (dense: 16 bytes; sparse: 8 bytes in .x/.y and the metadata dword in .z)
// and the four E8M0 scales of the step's blocks (byte j = block 4 ks + j).
struct SlotStep {
  uint4 c[2];
  uint32_t s;
};

template <int KIND>
__device__ __forceinline__ void load_slot_mx(SlotStep& d, const SlotBuf& b, int64_t r, int64_t R, int ks, int half,
                                             int nblk, int K) {
  if (KIND == 0) return;
  const int wp = min(128, K - 128 * ks);
  const int64_t pr = (int64_t)ks * R;
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    const int j = 2 * sub + half;
    const bool ok = 4 * ks + j < nblk;
    if (KIND == kSlotDense) {
      d.c[sub] = ok ? *reinterpret_cast<const uint4*>(b.c + pr * 64 + r * (wp / 2) + 16 * j) : make_uint4(0u, 0u, 0u, 0u);
    } else {
      const uint2 c = ok ? *reinterpret_cast<const uint2*>(b.c + pr * 32 + r * (wp / 4) + 8 * j) : make_uint2(0u, 0u);
      const uint32_t m = ok ? *reinterpret_cast<const uint32_t*>(b.m + pr * 16 + r * (wp / 8) + 4 * j) : 0x44444444u;
      d.c[sub] = make_uint4(c.x, c.y, m, 0u);
    }
  }
  const uint8_t* sr = b.s + pr * 4 + r * (wp / 32);
  d.s = 0u;
#pragma unroll
  for (int j = 0; j < 4; ++j) d.s |= (uint32_t)(4 * ks + j < nblk ? sr[j] : 127u) << (8 * j);
}

template <int KIND>
__device__ __forceinline__ v8i slot_operand(const uint4& c) {
  if (KIND == kSlotDense) return as_operand(c);
  return as_operand(expand_block<KIND>(make_uint2(c.x, c.y), c.z));
}

template <int SUB, int KIND>
__device__ __forceinline__ void mma_slot(v16f (&acc)[8], const v8i (&b)[8], const SlotStep& a, const uint32_t (&bw)[4],
                                         int half) {
  if (KIND == 0) return;
  const v8i op = slot_operand<KIND>(a.c[SUB]);
  const uint32_t sa = a.s >> (8 * half);
#pragma unroll
  for (int f = 0; f < 8; ++f) {
    if (f & 1) acc[f] = mfma_fp4<2 * SUB, 2 + SUB>(op, b[f], acc[f], sa, bw[f >> 1]);
    else       acc[f] = mfma_fp4<2 * SUB, SUB>(op, b[f], acc[f], sa, bw[f >> 1]);
  }
}

template <int K1, int K2>
__device__ __forceinline__ void step_slots(v16f (&acc)[8], const SlotStep& a1, const SlotStep& a2, const uint8_t* lw,
                                           const uint8_t* ls, int lane) {
  const int half = lane >> 5, col = lane & 31;
  uint32_t bw[4];
  const uint4 q = *reinterpret_cast<const uint4*>(ls + (2 * col + half) * 16);
  bw[0] = q.x; bw[1] = q.y; bw[2] = q.z; bw[3] = q.w;
#pragma unroll
  for (int sub = 0; sub < 2; ++sub) {
    v8i b[8];
#pragma unroll
    for (int f = 0; f < 8; ++f)
      b[f] = as_operand(*reinterpret_cast<const uint4*>(lw + (f * 32 + col) * kLdsStride + 32 * sub + 16 * half));
    if (sub == 0) {
      mma_slot<0, K1>(acc, b, a1, bw, half);
      mma_slot<0, K2>(acc, b, a2, bw, half);
    } else {
      mma_slot<1, K1>(acc, b, a1, bw, half);
      mma_slot<1, K2>(acc, b, a2, bw, half);
    }
  }
}

template <int K1, int K2, typename OutT>
__global__ __launch_bounds__(256) void k_linear_slots_mx(SlotBuf p1, SlotBuf p2, int64_t M, const uint8_t* wc,
                                                         const uint8_t* ws, int N, int K, OutT* Y, int64_t ldy,
                                                         int gx, int gy) {
  constexpr int NF = 8, BN = 256;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * BN * kLdsStride + 2 * 64 * 16];
  uint8_t* const lds_w = lds;
  uint8_t* const lds_s = lds + 2 * BN * kLdsStride;
  constexpr int SREC = 64 * 16;
  int mt, nt;
  tile_of(blockIdx.x, gx, gy, mt, nt);
  const int n0 = nt * BN;
  const int64_t row_lo = (int64_t)mt * kBM;
  const int64_t row_hi = row_lo + kBM < M ? row_lo + kBM : M;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5;
  const int nblk = K / 32, nks = (K + kBK - 1) / kBK;
  int64_t r = row_lo + wave * 32 + (lane & 31);
  if (r >= row_hi) r = row_hi - 1;   // clamp: loads stay in bounds, stores are masked

  v16f acc[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[f][e] = 0.0f;

  // the double-buffered pipeline of tile_mx: step ks computes from buffer
  // ks & 1 while the weight tile of ks + 1 goes to the other buffer and the
  // loads of ks + 2 are issued
  SlotStep a0[2], a1[2];
  WStep<NF> wn;
  const int last = nks - 1;
  load_w<NF, false>(wn, wc, ws, n0, N, K, 0, nblk);
  load_slot_mx<K1>(a0[0], p1, r, M, 0, half, nblk, K);
  load_slot_mx<K2>(a0[1], p2, r, M, 0, half, nblk, K);
  store_w<NF>(wn, lds_w, lds_s);
  load_w<NF, false>(wn, wc, ws, n0, N, K, min(1, last), nblk);
  load_slot_mx<K1>(a1[0], p1, r, M, min(1, last), half, nblk, K);
  load_slot_mx<K2>(a1[1], p2, r, M, min(1, last), half, nblk, K);
  int ks = 0;
  for (; ks + 1 < nks; ks += 2) {
    __syncthreads();
    step_slots<K1, K2>(acc, a0[0], a0[1], lds_w, lds_s, lane);
    store_w<NF>(wn, lds_w + BN * kLdsStride, lds_s + SREC);
    load_w<NF, false>(wn, wc, ws, n0, N, K, min(ks + 2, last), nblk);
    load_slot_mx<K1>(a0[0], p1, r, M, min(ks + 2, last), half, nblk, K);
    load_slot_mx<K2>(a0[1], p2, r, M, min(ks + 2, last), half, nblk, K);
    __syncthreads();
    step_slots<K1, K2>(acc, a1[0], a1[1], lds_w + BN * kLdsStride, lds_s + SREC, lane);
    store_w<NF>(wn, lds_w, lds_s);
    load_w<NF, false>(wn, wc, ws, n0, N, K, min(ks + 3, last), nblk);
    load_slot_mx<K1>(a1[0], p1, r, M, min(ks + 3, last), half, nblk, K);
    load_slot_mx<K2>(a1[1], p2, r, M, min(ks + 3, last), half, nblk, K);
  }
  if (ks < nks) {
    __syncthreads();
    step_slots<K1, K2>(acc, a0[0], a0[1], lds_w, lds_s, lane);
  }
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int col = n0 + f * 32 + (lane & 31);
    if (col >= N) continue;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t row = row_lo + wave * 32 + 8 * (e / 4) + 4 * half + (e % 4);
      if (row < row_hi) store_out<OutT>(Y + row * ldy + col, acc[f][e]);
    }
  }
}

// NVFP4: one K step is one 32-position block; both operands are exactly
// dequantized to bf16 (see k_linear_nv).  A dense slot has two E4M3 scales
// per block (halves of 16), a sparse slot one.
struct SlotNv {
  uint4 c;      // dense: codes; sparse: codes in .x/.y, metadata in .z
  uint32_t s;   // scale byte(s)
};

template <int KIND>
__device__ __forceinline__ void load_slot_nv(SlotNv& d, const SlotBuf& b, int64_t r, int64_t R, int ks, int K) {
  if (KIND == 0) return;
  const int p = ks >> 2, j = ks & 3, wp = min(128, K - 128 * p);
  const int64_t pr = (int64_t)p * R;
  if (KIND == kSlotDense) {
    d.c = *reinterpret_cast<const uint4*>(b.c + pr * 64 + r * (wp / 2) + 16 * j);
    d.s = *reinterpret_cast<const uint16_t*>(b.s + pr * 8 + r * (wp / 16) + 2 * j);
  } else {
    const uint2 c = *reinterpret_cast<const uint2*>(b.c + pr * 32 + r * (wp / 4) + 8 * j);
    d.c = make_uint4(c.x, c.y, *reinterpret_cast<const uint32_t*>(b.m + pr * 16 + r * (wp / 8) + 4 * j), 0u);
    d.s = b.s[pr * 4 + r * (wp / 32) + j];
  }
}

// this lane's bf16 operand of sub-step t: K values 8 half + 16 t + 0..7
template <int KIND>
__device__ __forceinline__ bf16x8 slot_nv_operand(const SlotNv& a, int t, int half) {
  if (KIND == kSlotDense) {
    const uint32_t w[4] = {a.c.x, a.c.y, a.c.z, a.c.w};
    const float d = e4m3_value(t ? (a.s >> 8) & 0xFFu : a.s & 0xFFu);
    return as_bf16x8(dequant8_bf16(w[half + 2 * t], d));
  }
  const uint4 e = expand_block<KIND>(make_uint2(a.c.x, a.c.y), a.c.z);
  const uint32_t w[4] = {e.x, e.y, e.z, e.w};
  return as_bf16x8(dequant8_bf16(w[half + 2 * t], e4m3_value(a.s & 0xFFu)));
}

template <int K1, int K2>
__device__ __forceinline__ void step_slots_nv(v16f (&acc)[8], const SlotNv& a1, const SlotNv& a2, const uint8_t* lw,
                                              int lane) {
  const int half = lane >> 5, col = lane & 31;
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    bf16x8 b[8];
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const int row = f * 32 + col;
      b[f] = as_bf16x8(*reinterpret_cast<const uint4*>(lw + row * 64 + 16 * ((half + 2 * t) ^ swz_nv(row))));
    }
    if (K1 != 0) {
      const bf16x8 a = slot_nv_operand<K1>(a1, t, half);
#pragma unroll
      for (int f = 0; f < 8; ++f) acc[f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b[f], acc[f], 0, 0, 0);
    }
    if (K2 != 0) {
      const bf16x8 a = slot_nv_operand<K2>(a2, t, half);
#pragma unroll
      for (int f = 0; f < 8; ++f) acc[f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b[f], acc[f], 0, 0, 0);
    }
  }
}

template <int K1, int K2, typename OutT>
__global__ __launch_bounds__(256) void k_linear_slots_nv(SlotBuf p1, SlotBuf p2, const float* ts_x, int64_t M,
                                                         const uint8_t* wc, const uint8_t* ws, const float* ts_w,
                                                         int N, int K, OutT* Y, int64_t ldy, int gx, int gy) {
  constexpr int NF = 8, BN = 256;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * BN * 64];
  int mt, nt;
  tile_of(blockIdx.x, gx, gy, mt, nt);
  const int n0 = nt * BN;
  const int64_t row_lo = (int64_t)mt * kBM;
  const int64_t row_hi = row_lo + kBM < M ? row_lo + kBM : M;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5;
  const int nks = K / 32;
  int64_t r = row_lo + wave * 32 + (lane & 31);
  if (r >= row_hi) r = row_hi - 1;

  v16f acc[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[f][e] = 0.0f;

  SlotNv a0[2], a1[2];
  NvW wn;
  const int last = nks - 1;
  load_nv_w<NF>(wn, wc, ws, n0, N, K, 0);
  load_slot_nv<K1>(a0[0], p1, r, M, 0, K);
  load_slot_nv<K2>(a0[1], p2, r, M, 0, K);
  store_nv_w(wn, lds);
  load_nv_w<NF>(wn, wc, ws, n0, N, K, min(1, last));
  load_slot_nv<K1>(a1[0], p1, r, M, min(1, last), K);
  load_slot_nv<K2>(a1[1], p2, r, M, min(1, last), K);
  int ks = 0;
  for (; ks + 1 < nks; ks += 2) {
    __syncthreads();
    step_slots_nv<K1, K2>(acc, a0[0], a0[1], lds, lane);
    store_nv_w(wn, lds + BN * 64);
    load_nv_w<NF>(wn, wc, ws, n0, N, K, min(ks + 2, last));
    load_slot_nv<K1>(a0[0], p1, r, M, min(ks + 2, last), K);
    load_slot_nv<K2>(a0[1], p2, r, M, min(ks + 2, last), K);
    __syncthreads();
    step_slots_nv<K1, K2>(acc, a1[0], a1[1], lds + BN * 64, lane);
    store_nv_w(wn, lds);
    load_nv_w<NF>(wn, wc, ws, n0, N, K, min(ks + 3, last));
    load_slot_nv<K1>(a1[0], p1, r, M, min(ks + 3, last), K);
    load_slot_nv<K2>(a1[1], p2, r, M, min(ks + 3, last), K);
  }
  if (ks < nks) {
    __syncthreads();
    step_slots_nv<K1, K2>(acc, a0[0], a0[1], lds, lane);
  }
  const float scale = *ts_x * *ts_w;
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int col = n0 + f * 32 + (lane & 31);
    if (col >= N) continue;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t row = row_lo + wave * 32 + 8 * (e / 4) + 4 * half + (e % 4);
      if (row < row_hi) store_out<OutT>(Y + row * ldy + col, acc[f][e] * scale);
    }
  }
}

// ---------------------------------------------------------------------------
// HiF4 two-path GEMM (2:4 backbone + dense residual).  No matrix instruction
// takes HiF4, but every HiF4 value E6M2 * 2^(E1_8 + E1_16) * S1P2 has at most
// 6 significant bits and an exponent in [-50, 17], so both operands are
// dequantized exactly to bf16 and multiplied on v_mfma_f32_32x32x16_bf16, as
// in the NVFP4 kernel (one K step = one 32-position block, the weight tile
// dequantized once per workgroup into LDS).  A unit's 4 metadata bytes
// [E6M2, E1_8, E1_16 low, E1_16 high] sit at its even block's 2-byte slots.
// ---------------------------------------------------------------------------

// The unit metadata word of block j of panel row (pr, r).
__device__ __forceinline__ uint32_t hif4_word_at(const uint8_t* sc, int64_t pr, int64_t r, int wp, int j) {
  return *reinterpret_cast<const uint32_t*>(sc + (pr * 4 + r * (wp / 32) + (j & ~1)) * 2);
}

// Eight codes (dword q of block half hb of a unit) -> eight exact bf16 values.
__device__ __forceinline__ uint4 hif4_dequant8_bf16(uint32_t codes, uint32_t word, int hb, int q) {
  const float base = e6m2_value(word & 0xFFu);
  const int l2 = 4 * hb + q, l3 = 8 * hb + 2 * q;
  const int e8 = (int)((word >> (8 + l2)) & 1u);
  const float sc0 = base * exp2_int(e8 + (int)((word >> (16 + l3)) & 1u));
  const float sc1 = base * exp2_int(e8 + (int)((word >> (17 + l3)) & 1u));
  uint32_t o[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float sc = i < 2 ? sc0 : sc1;
    const float a = s1p2_value((codes >> (8 * i)) & 0xFu, sc), b = s1p2_value((codes >> (8 * i + 4)) & 0xFu, sc);
    o[i] = __builtin_amdgcn_perm(__float_as_uint(b), __float_as_uint(a), 0x07060302u);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}

struct HfA {           // one lane's activation data for one block
  uint4 dn;            // residual codes
  uint2 spc;           // compressed backbone codes
  uint32_t spm;        // backbone metadata (2:4)
  uint32_t sw, dw;     // backbone and residual unit words
};

struct HfW {           // one thread's weight row for one block
  uint4 codes;
  uint32_t word;
};

__device__ __forceinline__ void load_hf_a(HfA& s, const ARow& a, int ks, int K) {
  const int p = ks >> 2, j = ks & 3, wp = min(128, K - 128 * p);
  const int64_t pr = (int64_t)p * a.R;
  s.dn = *reinterpret_cast<const uint4*>(a.dn + pr * 64 + a.r * (wp / 2) + 16 * j);
  s.spc = *reinterpret_cast<const uint2*>(a.spc + pr * 32 + a.r * (wp / 4) + 8 * j);
  s.spm = *reinterpret_cast<const uint32_t*>(a.spm + pr * 16 + a.r * (wp / 8) + 4 * j);
  s.sw = hif4_word_at(a.sps, pr, a.r, wp, j);
  s.dw = hif4_word_at(a.dns, pr, a.r, wp, j);
}

__device__ __forceinline__ void load_hf_w(HfW& w, const uint8_t* wc, const uint8_t* ws, int n0, int N, int K, int ks) {
  const int p = ks >> 2, j = ks & 3, wp = min(128, K - 128 * p);
  const int64_t pn = (int64_t)p * N;
  const int n = min(n0 + (int)threadIdx.x, N - 1);
  w.codes = *reinterpret_cast<const uint4*>(wc + pn * 64 + (int64_t)n * (wp / 2) + 16 * j);
  w.word = hif4_word_at(ws, pn, n, wp, j);
}

__device__ __forceinline__ void store_hf_w(const HfW& w, uint8_t* lds, int hb) {
  const int row = threadIdx.x;
  const uint32_t c[4] = {w.codes.x, w.codes.y, w.codes.z, w.codes.w};
#pragma unroll
  for (int q = 0; q < 4; ++q)
    *reinterpret_cast<uint4*>(lds + row * 64 + 16 * (q ^ swz_nv(row))) = hif4_dequant8_bf16(c[q], w.word, hb, q);
}

__device__ __forceinline__ void step_hf(v16f (&acc)[8], const HfA& a, int hb, const uint8_t* lw, int lane) {
  const int half = lane >> 5, col = lane & 31;
  const uint4 sp = expand_block<24>(a.spc, a.spm);
  const uint32_t spw[4] = {sp.x, sp.y, sp.z, sp.w};
  const uint32_t dnw[4] = {a.dn.x, a.dn.y, a.dn.z, a.dn.w};
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int q = half + 2 * t;   // K values 8 q .. 8 q + 7 of the block
    const bf16x8 asp = as_bf16x8(hif4_dequant8_bf16(spw[q], a.sw, hb, q));
    const bf16x8 adn = as_bf16x8(hif4_dequant8_bf16(dnw[q], a.dw, hb, q));
    bf16x8 b[8];
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const int row = f * 32 + col;
      b[f] = as_bf16x8(*reinterpret_cast<const uint4*>(lw + row * 64 + 16 * (q ^ swz_nv(row))));
    }
#pragma unroll
    for (int f = 0; f < 8; ++f) acc[f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(asp, b[f], acc[f], 0, 0, 0);
#pragma unroll
    for (int f = 0; f < 8; ++f) acc[f] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(adn, b[f], acc[f], 0, 0, 0);
  }
}

template <typename OutT>
__global__ __launch_bounds__(256) void k_linear_hif4(const uint8_t* sp_codes, const uint8_t* sp_meta,
                                                     const uint8_t* sp_scale, const uint8_t* dn_codes,
                                                     const uint8_t* dn_scale, int64_t M, const uint8_t* wc,
                                                     const uint8_t* ws, int N, int K, OutT* Y, int64_t ldy, int gx,
                                                     int gy) {
  constexpr int NF = 8, BN = 256;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * BN * 64];
  int mt, nt;
  tile_of(blockIdx.x, gx, gy, mt, nt);
  const int n0 = nt * BN;
  const int64_t row_lo = (int64_t)mt * kBM;
  const int64_t row_hi = row_lo + kBM < M ? row_lo + kBM : M;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, half = lane >> 5;
  const int nks = K / 32;
  int64_t orow = row_lo + wave * 32 + (lane & 31);
  if (orow >= row_hi) orow = row_hi - 1;
  ARow a;
  a.r = orow;
  a.R = M;
  a.dn = dn_codes;
  a.spc = sp_codes;
  a.spm = sp_meta;
  a.dns = dn_scale;
  a.sps = sp_scale;

  v16f acc[NF];
#pragma unroll
  for (int f = 0; f < NF; ++f)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[f][e] = 0.0f;

  // the double-buffered pipeline of k_linear_nv; block ks is half ks & 1 of its unit
  HfA a0, a1;
  HfW wn;
  const int last = nks - 1;
  load_hf_w(wn, wc, ws, n0, N, K, 0);
  load_hf_a(a0, a, 0, K);
  store_hf_w(wn, lds, 0);
  load_hf_w(wn, wc, ws, n0, N, K, min(1, last));
  load_hf_a(a1, a, min(1, last), K);
  int ks = 0;
  for (; ks + 1 < nks; ks += 2) {   // nks is even: blocks ks, ks + 1 are the halves of one unit
    __syncthreads();
    step_hf(acc, a0, 0, lds, lane);
    store_hf_w(wn, lds + BN * 64, 1);
    load_hf_w(wn, wc, ws, n0, N, K, min(ks + 2, last));
    load_hf_a(a0, a, min(ks + 2, last), K);
    __syncthreads();
    step_hf(acc, a1, 1, lds + BN * 64, lane);
    store_hf_w(wn, lds, 0);
    load_hf_w(wn, wc, ws, n0, N, K, min(ks + 3, last));
    load_hf_a(a1, a, min(ks + 3, last), K);
  }
#pragma unroll
  for (int f = 0; f < NF; ++f) {
    const int col = n0 + f * 32 + (lane & 31);
    if (col >= N) continue;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t row = row_lo + wave * 32 + 8 * (e / 4) + 4 * half + (e % 4);
      if (row < row_hi) store_out<OutT>(Y + row * ldy + col, acc[f][e]);
    }
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers
// ---------------------------------------------------------------------------

// Compute units of the current device (queried once per device).
static int device_cus() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (cache[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

// Work units of the persistent kernel: whole tiles, with a last round that
// would be at most half full run as twice as many half tiles.
struct PersistPlan {
  int grid, full, halves;
};

static PersistPlan persist_plan(int gx, int gy) {
  const int tiles = gx * gy, cus = device_cus();
  PersistPlan p{tiles < cus ? tiles : cus, tiles, 0};
  const int r = tiles % p.grid;
  if (tiles > p.grid && r > 0 && 2 * r <= p.grid) {
    p.full = tiles - r;
    p.halves = 2 * r;
  }
  return p;
}

template <int NF, int PAT, bool SDW, typename OutT>
static hipError_t go_linear(const uint8_t* spc, const uint8_t* spm, const uint8_t* sps, const uint8_t* dnc,
                            const uint8_t* dns, int64_t M, const uint8_t* wc, const uint8_t* ws, int N, int K,
                            void* Y, int64_t ldy, hipStream_t st) {
  const int gx = (N + 32 * NF - 1) / (32 * NF), gy = (int)((M + kBM - 1) / kBM);
  if constexpr (SDW && NF == 8) {
    const PersistPlan pl = persist_plan(gx, gy);
    k_linear_mx_persist<PAT, OutT><<<dim3((unsigned)pl.grid), dim3(256), 0, st>>>(
        spc, spm, sps, dnc, dns, M, wc, ws, N, K, reinterpret_cast<OutT*>(Y), ldy, gx, gy, pl.full, pl.halves);
  } else {
    k_linear_mx<NF, PAT, SDW, OutT><<<dim3((unsigned)(gx * gy)), dim3(256), 0, st>>>(
        spc, spm, sps, dnc, dns, M, wc, ws, N, K, reinterpret_cast<OutT*>(Y), ldy, gx, gy);
  }
  return hipGetLastError();
}

template <int NF, int PAT, bool SDW>
static hipError_t go_linear_dt(int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps,
                               const uint8_t* dnc, const uint8_t* dns, int64_t M, const uint8_t* wc,
                               const uint8_t* ws, int N, int K, void* Y, int64_t ldy, hipStream_t st) {
  if (ydt == 2) return go_linear<NF, PAT, SDW, float>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
  if (ydt == 1) return go_linear<NF, PAT, SDW, _Float16>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
  return go_linear<NF, PAT, SDW, uint16_t>(spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
}

// The persistent interleaved kernel on a dense backbone copy (pattern 0).
template <typename OutT>
static hipError_t go_dense_backbone(const uint8_t* spd, const uint8_t* sps, const uint8_t* dnc, const uint8_t* dns,
                                    int64_t M, const uint8_t* wc, const uint8_t* ws, int N, int K, void* Y,
                                    int64_t ldy, hipStream_t st) {
  const int gx = (N + 255) / 256, gy = (int)((M + kBM - 1) / kBM);
  const PersistPlan pl = persist_plan(gx, gy);
  k_linear_mx_persist<0, OutT><<<dim3((unsigned)pl.grid), dim3(256), 0, st>>>(
      spd, nullptr, sps, dnc, dns, M, wc, ws, N, K, reinterpret_cast<OutT*>(Y), ldy, gx, gy, pl.full, pl.halves);
  return hipGetLastError();
}

// spd (optional): the backbone's dense copy; used by the main kernel (K a
// multiple of 128, M beyond the small-M kernel's range), which then skips the
// expansion.
hipError_t launch_linear_mx(int pat, int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps,
                            const uint8_t* dnc, const uint8_t* dns, int64_t M, const uint8_t* wc, const uint8_t* ws,
                            int N, int K, void* Y, int64_t ldy, const uint8_t* spd, hipStream_t st) {
  const bool sdw = (K % kBK) == 0;
  constexpr int NF = 8;
  if (spd && sdw && !use_skinny(M, N, K)) {
    if (ydt == 2) return go_dense_backbone<float>(spd, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
    if (ydt == 1) return go_dense_backbone<_Float16>(spd, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
    return go_dense_backbone<uint16_t>(spd, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
  }
  if (use_skinny(M, N, K)) {
    if (spc == nullptr)   // the backbone exists as its dense copy only
      return go_skinny_dt<0>(ydt, spd, nullptr, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
    return pat == 24 ? go_skinny_dt<24>(ydt, spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st)
                     : go_skinny_dt<48>(ydt, spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
  }
  if (spc == nullptr) return hipErrorInvalidValue;   // rejected by the C ABI (K not a multiple of 128)
  if (pat == 24) {
    return sdw ? go_linear_dt<NF, 24, true>(ydt, spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st)
               : go_linear_dt<NF, 24, false>(ydt, spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
  }
  return sdw ? go_linear_dt<NF, 48, true>(ydt, spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st)
             : go_linear_dt<NF, 48, false>(ydt, spc, spm, sps, dnc, dns, M, wc, ws, N, K, Y, ldy, st);
}

template <int NF, int PAT, bool SDW, typename OutT>
static hipError_t go_grouped(const uint8_t* spc, const uint8_t* spm, const uint8_t* sps, const uint8_t* dnc,
                             const uint8_t* dns, const int32_t* ridx, int64_t act_rows, const int32_t* offs, int E,
                             int64_t total, const uint8_t* wc, const uint8_t* ws, int N, int K, void* Y, int64_t ldy,
                             hipStream_t st) {
  // upper bound on the number of 128-row tiles over all experts
  const int64_t items = (total + kBM - 1) / kBM + E;
  const int gx = (N + 32 * NF - 1) / (32 * NF);
  if ((int64_t)gx * items > (int64_t)INT32_MAX) return hipErrorInvalidValue;
  if constexpr (SDW && NF == 8) {
    const int64_t bound = (int64_t)gx * items, cus = device_cus();
    const unsigned g = (unsigned)(bound < cus ? bound : cus);
    if (ridx)
      k_linear_mx_grouped_persist<PAT, OutT, true><<<dim3(g), dim3(256), 0, st>>>(
          spc, spm, sps, dnc, dns, ridx, act_rows, offs, E, wc, ws, N, K, reinterpret_cast<OutT*>(Y), ldy, gx);
    else
      k_linear_mx_grouped_persist<PAT, OutT, false><<<dim3(g), dim3(256), 0, st>>>(
          spc, spm, sps, dnc, dns, ridx, act_rows, offs, E, wc, ws, N, K, reinterpret_cast<OutT*>(Y), ldy, gx);
    return hipGetLastError();
  }
  dim3 grid((unsigned)(gx * items)), block(256);
  k_linear_mx_grouped<NF, PAT, SDW, OutT><<<grid, block, 0, st>>>(spc, spm, sps, dnc, dns, ridx, act_rows, offs, E,
                                                                  wc, ws, N, K, reinterpret_cast<OutT*>(Y), ldy, gx);
  return hipGetLastError();
}

template <int NF, int PAT, bool SDW>
static hipError_t go_grouped_dt(int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps,
                                const uint8_t* dnc, const uint8_t* dns, const int32_t* ridx, int64_t act_rows,
                                const int32_t* offs, int E, int64_t total, const uint8_t* wc, const uint8_t* ws, int N,
                                int K, void* Y, int64_t ldy, hipStream_t st) {
  if (ydt == 2)
    return go_grouped<NF, PAT, SDW, float>(spc, spm, sps, dnc, dns, ridx, act_rows, offs, E, total, wc, ws, N, K, Y, ldy, st);
  if (ydt == 1)
    return go_grouped<NF, PAT, SDW, _Float16>(spc, spm, sps, dnc, dns, ridx, act_rows, offs, E, total, wc, ws, N, K, Y, ldy,
                                              st);
  return go_grouped<NF, PAT, SDW, uint16_t>(spc, spm, sps, dnc, dns, ridx, act_rows, offs, E, total, wc, ws, N, K, Y, ldy,
                                            st);
}

// spd (optional): the backbone's dense copy, read instead of expanding the
// compressed backbone when K is a multiple of 128.
hipError_t launch_linear_mx_grouped(int pat, int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps,
                                    const uint8_t* dnc, const uint8_t* dns, const int32_t* ridx, int64_t act_rows,
                                    const int32_t* offs, int E, int64_t total, const uint8_t* wc, const uint8_t* ws,
                                    int N, int K, void* Y, int64_t ldy, const uint8_t* spd, hipStream_t st) {
  const bool sdw = (K % kBK) == 0;
  constexpr int NF = 8;
  if (spd && sdw)
    return go_grouped_dt<NF, 0, true>(ydt, spd, nullptr, sps, dnc, dns, ridx, act_rows, offs, E, total, wc, ws, N, K,
                                      Y, ldy, st);
  if (pat == 24) {
    return sdw ? go_grouped_dt<NF, 24, true>(ydt, spc, spm, sps, dnc, dns, ridx, act_rows, offs, E, total, wc, ws, N, K, Y,
                                             ldy, st)
               : go_grouped_dt<NF, 24, false>(ydt, spc, spm, sps, dnc, dns, ridx, act_rows, offs, E, total, wc, ws, N, K, Y,
                                              ldy, st);
  }
  return sdw ? go_grouped_dt<NF, 48, true>(ydt, spc, spm, sps, dnc, dns, ridx, act_rows, offs, E, total, wc, ws, N, K, Y, ldy,
                                           st)
             : go_grouped_dt<NF, 48, false>(ydt, spc, spm, sps, dnc, dns, ridx, act_rows, offs, E, total, wc, ws, N, K, Y, ldy,
                                            st);
}


template <int K1, int K2, typename OutT>
static hipError_t go_slots(bool nv, const SlotBuf& p1, const SlotBuf& p2, const float* tsx, int64_t M,
                           const uint8_t* wc, const uint8_t* ws, const float* tsw, int N, int K, void* Y, int64_t ldy,
                           hipStream_t st) {
  const int gx = (N + 255) / 256, gy = (int)((M + kBM - 1) / kBM);
  const dim3 grid((unsigned)(gx * gy)), block(256);
  if (nv)
    k_linear_slots_nv<K1, K2, OutT><<<grid, block, 0, st>>>(p1, p2, tsx, M, wc, ws, tsw, N, K,
                                                            reinterpret_cast<OutT*>(Y), ldy, gx, gy);
  else
    k_linear_slots_mx<K1, K2, OutT><<<grid, block, 0, st>>>(p1, p2, M, wc, ws, N, K, reinterpret_cast<OutT*>(Y), ldy,
                                                            gx, gy);
  return hipGetLastError();
}

template <int K1, int K2>
static hipError_t go_slots_dt(int ydt, bool nv, const SlotBuf& p1, const SlotBuf& p2, const float* tsx, int64_t M,
                              const uint8_t* wc, const uint8_t* ws, const float* tsw, int N, int K, void* Y,
                              int64_t ldy, hipStream_t st) {
  if (ydt == 2) return go_slots<K1, K2, float>(nv, p1, p2, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
  if (ydt == 1) return go_slots<K1, K2, _Float16>(nv, p1, p2, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
  return go_slots<K1, K2, uint16_t>(nv, p1, p2, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
}

// Path combinations (modes 1-4 of the C interface): 1 sparse, 2 dense (RTN),
// 3 dense + dense, 4 sparse + sparse.  pat: 24 or 48 (the sparse metadata
// layout).  nv: NVFP4 (the weight's sparse view `ws` serves every path: its
// per-16 dense view holds the same values).
hipError_t launch_linear_slots(int mode, int pat, int ydt, bool nv, const uint8_t* c1, const uint8_t* m1,
                               const uint8_t* s1, const uint8_t* c2, const uint8_t* m2, const uint8_t* s2,
                               const float* tsx, int64_t M, const uint8_t* wc, const uint8_t* ws, const float* tsw,
                               int N, int K, void* Y, int64_t ldy, hipStream_t st) {
  const SlotBuf p1{c1, m1, s1}, p2{c2, m2, s2};
  const bool p24 = pat == 24;
  switch (mode) {
    case 1: return p24 ? go_slots_dt<24, 0>(ydt, nv, p1, p2, tsx, M, wc, ws, tsw, N, K, Y, ldy, st)
                       : go_slots_dt<48, 0>(ydt, nv, p1, p2, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
    case 2: return go_slots_dt<0, kSlotDense>(ydt, nv, p1, p2, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
    case 3: return go_slots_dt<kSlotDense, kSlotDense>(ydt, nv, p1, p2, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
    case 4: return p24 ? go_slots_dt<24, 24>(ydt, nv, p1, p2, tsx, M, wc, ws, tsw, N, K, Y, ldy, st)
                       : go_slots_dt<48, 48>(ydt, nv, p1, p2, tsx, M, wc, ws, tsw, N, K, Y, ldy, st);
    default: return hipErrorInvalidValue;
  }
}


// HiF4 (2:4 backbone, K a multiple of 64).
hipError_t launch_linear_hif4(int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps, const uint8_t* dnc,
                              const uint8_t* dns, int64_t M, const uint8_t* wc, const uint8_t* ws, int N, int K,
                              void* Y, int64_t ldy, hipStream_t st) {
  const int gx = (N + 255) / 256, gy = (int)((M + kBM - 1) / kBM);
  const dim3 grid((unsigned)(gx * gy)), block(256);
  if (ydt == 2)
    k_linear_hif4<float><<<grid, block, 0, st>>>(spc, spm, sps, dnc, dns, M, wc, ws, N, K,
                                                 reinterpret_cast<float*>(Y), ldy, gx, gy);
  else if (ydt == 1)
    k_linear_hif4<_Float16><<<grid, block, 0, st>>>(spc, spm, sps, dnc, dns, M, wc, ws, N, K,
                                                    reinterpret_cast<_Float16*>(Y), ldy, gx, gy);
  else
    k_linear_hif4<uint16_t><<<grid, block, 0, st>>>(spc, spm, sps, dnc, dns, M, wc, ws, N, K,
                                                    reinterpret_cast<uint16_t*>(Y), ldy, gx, gy);
  return hipGetLastError();
}

}  // namespace sharq
