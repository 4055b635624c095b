// Block-level device code of the SharQ activation preparation (Sec. 3.4,
// "Fused sparse-residual preparation"; Sec. 3.3 eqs. "dynamic-mask",
// "sharq-quantized-backbone", "sharq-residual"), shared by the preparation
// kernels and the small-M GEMM with the preparation in its prologue: the N:M
// selection, the MXFP4 and NVFP4 block quantizers with the residual, the
// RMSNorm reductions, the output addressing and the row loaders.  Compiled
// without contraction into fused multiply-add, like its users.
#pragma once

#include "sharq_device.hpp"

#pragma clang fp contract(off)

namespace sharq {

// ---------------------------------------------------------------------------
// N:M selection inside one block
// ---------------------------------------------------------------------------

// Lane masks.  A comparison over the wavefront is one vector instruction that
// leaves a 64-bit mask in scalar registers; logic on masks runs on the
// scalar unit, beside the vector work of the other wavefronts, and the masks
// drive per-lane selects directly.
typedef uint64_t lmask;

__device__ __forceinline__ lmask ge_mask(float a, float b) { return __builtin_amdgcn_ballot_w64(a >= b); }

// this lane's bit of m ? t : f
__device__ __forceinline__ float lsel(lmask m, float t, float f) {
  float r;
  asm("v_cndmask_b32_e64 %0, %1, %2, %3" : "=v"(r) : "v"(f), "v"(t), "s"(m));
  return r;
}

// 2 v + this lane's bit of m (the metadata is shifted in one bit at a time)
__device__ __forceinline__ uint32_t push_bit(uint32_t v, lmask m) {
  uint32_t r;
  lmask carry;
  asm("v_addc_co_u32_e64 %0, %1, %2, %2, %3" : "=v"(r), "=s"(carry) : "v"(v), "s"(m));
  return r;
}

__device__ __forceinline__ lmask maj3(lmask a, lmask b, lmask c) { return (a & b) | (c & (a | b)); }

// 2:4 on one group: keep masks of positions 0..3 (exactly two set per lane).
// Position p survives iff it beats at least two of the other three, where of
// p < q, p beats q iff |y_p| >= |y_q| (a tie goes to the lower index): six
// comparisons, then four majority votes on the scalar unit.
__device__ __forceinline__ void top2of4(float y0, float y1, float y2, float y3, lmask& k0, lmask& k1, lmask& k2,
                                        lmask& k3) {
  const float a0 = fabsf(y0), a1 = fabsf(y1), a2 = fabsf(y2), a3 = fabsf(y3);
  const lmask c01 = ge_mask(a0, a1), c02 = ge_mask(a0, a2), c03 = ge_mask(a0, a3);
  const lmask c12 = ge_mask(a1, a2), c13 = ge_mask(a1, a3), c23 = ge_mask(a2, a3);
  k0 = maj3(c01, c02, c03);
  k1 = maj3(~c01, c12, c13);
  k2 = maj3(~c02, ~c12, c23);
  k3 = maj3(~c03, ~c13, ~c23);
}

template <int SEL, class Q>
__device__ __forceinline__ void put_pair(const Q& qz, uint32_t& word, float a, float b) {
  word = qz.template enc2<SEL>(word, a, b);
}

template <class Q>
__device__ __forceinline__ void put_pair_dyn(const Q& qz, uint32_t& word, int sel, float a, float b) {
  switch (sel & 3) {
    case 0: put_pair<0>(qz, word, a, b); break;
    case 1: put_pair<1>(qz, word, a, b); break;
    case 2: put_pair<2>(qz, word, a, b); break;
    default: put_pair<3>(qz, word, a, b); break;
  }
}

// dequantized values of the two codes in byte `sel` of `word`
template <class Q>
__device__ __forceinline__ v2f get_pair_dyn(const Q& qz, uint32_t word, int sel) {
  switch (sel & 3) {
    case 0: return qz.template dec2<0>(word);
    case 1: return qz.template dec2<1>(word);
    case 2: return qz.template dec2<2>(word);
    default: return qz.template dec2<3>(word);
  }
}

// Backbone of one block for the 2:4 pattern.  Returns the residual in R:
// y minus the dequantized code at kept positions, y elsewhere.
template <class Q>
__device__ __forceinline__ void backbone_24(const float (&y)[32], const Q& qz, uint32_t (&codes)[2], uint32_t& meta,
                                            float (&R)[32]) {
  codes[0] = codes[1] = 0u;
  meta = 0u;
  // groups from the last to the first: the metadata is shifted in from its
  // top bit down
#pragma unroll
  for (int g = 7; g >= 0; --g) {
    const float y0 = y[4 * g], y1 = y[4 * g + 1], y2 = y[4 * g + 2], y3 = y[4 * g + 3];
    lmask k0, k1, k2, k3;
    top2of4(y0, y1, y2, y3, k0, k1, k2, k3);
    const float v0 = lsel(k0, y0, lsel(k1, y1, y2));   // first kept (ascending K)
    const float v1 = lsel(k3, y3, lsel(k2, y2, y1));   // second kept
    // nibble i0 | i1 << 2: i0 = 0, 1, 2 and i1 = 3, 2, 1 as above
    meta = push_bit(meta, k3 | k2);                    // bit 3: i1 >= 2
    meta = push_bit(meta, k3 | ~k2);                   // bit 2: i1 odd
    meta = push_bit(meta, ~(k0 | k1));                 // bit 1: i0 == 2
    meta = push_bit(meta, k1 & ~k0);                   // bit 0: i0 == 1
    // the other bytes of a codes dword are written by the groups that follow
    // in this loop, so the dword's first group may start from any register
    if ((g & 3) == 3) codes[g >> 2] = __float_as_uint(v0);
    put_pair_dyn(qz, codes[g >> 2], g, v0, v1);
    const v2f d = get_pair_dyn(qz, codes[g >> 2], g);
    const float r0 = v0 - d.x, r1 = v1 - d.y;
    R[4 * g + 0] = lsel(k0, r0, y0);
    R[4 * g + 1] = lsel(k1, lsel(k0, r1, r0), y1);
    R[4 * g + 2] = lsel(k2, lsel(k3, r0, r1), y2);
    R[4 * g + 3] = lsel(k3, r1, y3);
  }
}

// The 2:4 backbone together with its dense copy (codes at all 32 positions,
// dropped positions code 0).  Converting the kept values in place, with +0 at
// the dropped positions, gives the dense codes directly; decoding them gives
// the residual at every position at once: y minus the dequantized code where
// kept, y - 0 = y (signed zeros included) where dropped -- the same values as
// backbone_24.  The compressed codes and metadata are those of backbone_24.
template <class Q>
__device__ __forceinline__ void backbone_24_dense(const float (&y)[32], const Q& qz, uint32_t (&codes)[2],
                                                  uint32_t& meta, uint32_t (&dense)[4], float (&R)[32]) {
  codes[0] = codes[1] = 0u;
  meta = 0u;
#pragma unroll
  for (int g = 7; g >= 0; --g) {
    const float y0 = y[4 * g], y1 = y[4 * g + 1], y2 = y[4 * g + 2], y3 = y[4 * g + 3];
    lmask k0, k1, k2, k3;
    top2of4(y0, y1, y2, y3, k0, k1, k2, k3);
    const float v0 = lsel(k0, y0, lsel(k1, y1, y2));   // first kept (ascending K)
    const float v1 = lsel(k3, y3, lsel(k2, y2, y1));   // second kept
    meta = push_bit(meta, k3 | k2);
    meta = push_bit(meta, k3 | ~k2);
    meta = push_bit(meta, ~(k0 | k1));
    meta = push_bit(meta, k1 & ~k0);
    if ((g & 3) == 3) codes[g >> 2] = __float_as_uint(v0);
    put_pair_dyn(qz, codes[g >> 2], g, v0, v1);
    // group g is bytes 2 (g & 1) and 2 (g & 1) + 1 of dense dword g / 2; the
    // odd group comes first in this loop and may start from any register
    const float b0 = lsel(k0, y0, 0.0f), b1 = lsel(k1, y1, 0.0f);
    const float b2 = lsel(k2, y2, 0.0f), b3 = lsel(k3, y3, 0.0f);
    if (g & 1) dense[g >> 1] = __float_as_uint(b0);
    put_pair_dyn(qz, dense[g >> 1], 2 * (g & 1), b0, b1);
    put_pair_dyn(qz, dense[g >> 1], 2 * (g & 1) + 1, b2, b3);
    const v2f d01 = get_pair_dyn(qz, dense[g >> 1], 2 * (g & 1));
    const v2f d23 = get_pair_dyn(qz, dense[g >> 1], 2 * (g & 1) + 1);
    R[4 * g + 0] = y0 - d01.x;
    R[4 * g + 1] = y1 - d01.y;
    R[4 * g + 2] = y2 - d23.x;
    R[4 * g + 3] = y3 - d23.y;
  }
}

// The 2:4 backbone as its dense codes only (no compressed codes, no
// metadata): the kept values converted in place with +0 at the dropped
// positions, and the residual decoded from them as in backbone_24_dense.
template <class Q>
__device__ __forceinline__ void backbone_24_dense_only(const float (&y)[32], const Q& qz, uint32_t (&dense)[4],
                                                       float (&R)[32]) {
#pragma unroll
  for (int g = 7; g >= 0; --g) {
    const float y0 = y[4 * g], y1 = y[4 * g + 1], y2 = y[4 * g + 2], y3 = y[4 * g + 3];
    lmask k0, k1, k2, k3;
    top2of4(y0, y1, y2, y3, k0, k1, k2, k3);
    const float b0 = lsel(k0, y0, 0.0f), b1 = lsel(k1, y1, 0.0f);
    const float b2 = lsel(k2, y2, 0.0f), b3 = lsel(k3, y3, 0.0f);
    if (g & 1) dense[g >> 1] = __float_as_uint(b0);
    put_pair_dyn(qz, dense[g >> 1], 2 * (g & 1), b0, b1);
    put_pair_dyn(qz, dense[g >> 1], 2 * (g & 1) + 1, b2, b3);
    const v2f d01 = get_pair_dyn(qz, dense[g >> 1], 2 * (g & 1));
    const v2f d23 = get_pair_dyn(qz, dense[g >> 1], 2 * (g & 1) + 1);
    R[4 * g + 0] = y0 - d01.x;
    R[4 * g + 1] = y1 - d01.y;
    R[4 * g + 2] = y2 - d23.x;
    R[4 * g + 3] = y3 - d23.y;
  }
}

// Keep bits of one block (bit p = position p kept) from its metadata: 2:4
// nibbles i0 | i1 << 2 per group, or the 4:8 keep masks themselves.
template <int PAT>
__device__ __forceinline__ uint32_t keep_bits(uint32_t meta) {
  if (PAT != 24) return meta;
  uint32_t k = 0u;
#pragma unroll
  for (int g = 0; g < 8; ++g) {
    const uint32_t nib = (meta >> (4 * g)) & 0xFu;
    k |= ((1u << (nib & 3u)) | (1u << (nib >> 2))) << (4 * g);
  }
  return k;
}

// 4:8 selection on one group of 8: of p < q, p beats q iff |y_p| >= |y_q|
// (a tie goes to the lower index), and a position survives iff it beats at
// least 4 of the other 7.  One comparison per pair counts on both sides
// (beats[p] starts at p: the lower positions, which it beats unless they
// beat it), the eight counts held as the nibbles of one word.  Returns the
// 8-bit keep mask and b = y where kept, +0 where dropped.
__device__ __forceinline__ uint32_t select48(const float* e, float (&b)[8]) {
  float a[8];
#pragma unroll
  for (int p = 0; p < 8; ++p) a[p] = fabsf(e[p]);
  // the eight counts as the nibbles of one word (nibble p = beats[p], 0..7 at
  // every point, so no nibble borrows or carries); a decided pair adds +1 to
  // nibble p and -1 to nibble q in one constant, two pairs per add
  uint32_t W = 0x76543210u, pend = 0u;
  int n = 0;
#pragma unroll
  for (int p = 0; p < 8; ++p)
#pragma unroll
    for (int q = p + 1; q < 8; ++q) {
      const uint32_t d = a[p] >= a[q] ? (1u << (4 * p)) - (1u << (4 * q)) : 0u;
      if (++n & 1) {
        pend = d;
      } else {
        W += pend + d;
      }
    }
  // 28 pairs: every increment added.  Position p survives iff bit 2 of its
  // nibble is set (beats[p] >= 4).
  uint32_t m = (W >> 2) & 0x11111111u;
  m = (m | (m >> 3)) & 0x03030303u;
  m = (m | (m >> 6)) & 0x000F000Fu;
  const uint32_t mask = (m | (m >> 12)) & 0xFFu;
#pragma unroll
  for (int p = 0; p < 8; ++p)
    b[p] = __uint_as_float(__float_as_uint(e[p]) & (uint32_t)((int32_t)(W << (29 - 4 * p)) >> 31));
  return mask;
}

// The four kept codes of a group (exactly four bits of mask set) out of its
// dense dword (code of position p in nibble p), packed in ascending position,
// low nibble first: the nibbles are spread to one byte per position, the
// kept bytes gathered by one byte permute, and the bytes packed back.
__device__ __forceinline__ uint32_t compact48(uint32_t dense, uint32_t mask) {
  const uint32_t lo = dense & 0x0F0F0F0Fu;          // positions 0, 2, 4, 6
  const uint32_t hi = (dense >> 4) & 0x0F0F0F0Fu;   // positions 1, 3, 5, 7
  // perm(s0, s1, sel): selector 0-3 takes byte k of s1, 4-7 byte k - 4 of s0
  const uint32_t q0 = __builtin_amdgcn_perm(hi, lo, 0x05010400u);   // positions 0..3, one per byte
  const uint32_t q1 = __builtin_amdgcn_perm(hi, lo, 0x07030602u);   // positions 4..7
  uint32_t m = mask, sel = 0u;
#pragma unroll
  for (int s = 0; s < 4; ++s) {
    sel |= (uint32_t)__builtin_ctz(m) << (8 * s);
    m &= m - 1u;
  }
  const uint32_t c = __builtin_amdgcn_perm(q1, q0, sel);   // kept codes k0..k3, one per byte
  const uint32_t t = c | (c >> 4);                          // k0 | k1 << 4 in byte 0, k2 | k3 << 4 in byte 2
  return (t & 0xFFu) | ((t >> 8) & 0xFF00u);
}

template <class Q>
__device__ __forceinline__ void dense_group8(const Q& qz, const float (&b)[8], const float* y, uint32_t& word,
                                             float* R);

// Backbone of one block for the 4:8 pattern (keep mask metadata): each group
// is converted in place (kept values, +0 where dropped), its residual taken
// against that, and the kept codes gathered from the dense dword.
template <class Q>
__device__ __forceinline__ void backbone_48(const float (&y)[32], const Q& qz, uint32_t (&codes)[2], uint32_t& meta,
                                            float (&R)[32]) {
  codes[0] = codes[1] = 0u;
  meta = 0u;
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    float b[8];
    const uint32_t mask = select48(y + 8 * g, b);
    meta |= mask << (8 * g);
    uint32_t dense;
    dense_group8(qz, b, y + 8 * g, dense, R + 8 * g);
    codes[g >> 1] |= compact48(dense, mask) << (16 * (g & 1));
  }
}

// Dense codes of one group of 8 (b: kept values, +0 where dropped) into one
// dword, low nibble first in ascending K, and the group's residual
// y - dequant(code): y itself where dropped (y - (+0) = y, signed zeros
// included).
template <class Q>
__device__ __forceinline__ void dense_group8(const Q& qz, const float (&b)[8], const float* y, uint32_t& word,
                                             float* R) {
  word = __float_as_uint(b[0]);   // every byte is overwritten below
  put_pair<0>(qz, word, b[0], b[1]);
  put_pair<1>(qz, word, b[2], b[3]);
  put_pair<2>(qz, word, b[4], b[5]);
  put_pair<3>(qz, word, b[6], b[7]);
  const v2f d0 = qz.template dec2<0>(word), d1 = qz.template dec2<1>(word);
  const v2f d2 = qz.template dec2<2>(word), d3 = qz.template dec2<3>(word);
  R[0] = y[0] - d0.x;
  R[1] = y[1] - d0.y;
  R[2] = y[2] - d1.x;
  R[3] = y[3] - d1.y;
  R[4] = y[4] - d2.x;
  R[5] = y[5] - d2.y;
  R[6] = y[6] - d3.x;
  R[7] = y[7] - d3.y;
}

// The backbone of one 4:8 block as its dense codes alone (dropped positions
// +0, so code 0), and the residual: backbone_48 without the compressed codes
// and the metadata.
template <class Q>
__device__ __forceinline__ void backbone_48_dense_only(const float (&y)[32], const Q& qz, uint32_t (&dense)[4],
                                                       float (&R)[32]) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    float b[8];
    select48(y + 8 * g, b);
    dense_group8(qz, b, y + 8 * g, dense[g], R + 8 * g);
  }
}

// The same for 4:8 in pairs: the 2:4 selection on the pair scores
// max(|y_2i|, |y_2i+1|), whole pairs kept (backbone_48p's selection).
template <class Q>
__device__ __forceinline__ void backbone_48p_dense_only(const float (&y)[32], const Q& qz, uint32_t (&dense)[4],
                                                        float (&R)[32]) {
#pragma unroll
  for (int g = 0; g < 4; ++g) {
    const float* e = y + 8 * g;
    const float s0 = fmaxf(fabsf(e[0]), fabsf(e[1])), s1 = fmaxf(fabsf(e[2]), fabsf(e[3]));
    const float s2 = fmaxf(fabsf(e[4]), fabsf(e[5])), s3 = fmaxf(fabsf(e[6]), fabsf(e[7]));
    lmask p0, p1, p2, p3;
    top2of4(s0, s1, s2, s3, p0, p1, p2, p3);
    const float b[8] = {lsel(p0, e[0], 0.0f), lsel(p0, e[1], 0.0f), lsel(p1, e[2], 0.0f), lsel(p1, e[3], 0.0f),
                        lsel(p2, e[4], 0.0f), lsel(p2, e[5], 0.0f), lsel(p3, e[6], 0.0f), lsel(p3, e[7], 0.0f)};
    dense_group8(qz, b, e, dense[g], R + 8 * g);
  }
}

// Backbone of one block for NVFP4's 4:8 in pairs (App. A.1.4): the 8
// positions of a group are 4 adjacent pairs and the 2 pairs with the largest
// scores max(|y_2i|, |y_2i+1|) survive, a tie going to the lower pair -- the
// 2:4 selection applied to the pair scores.  The group maximum lies in a kept
// pair, so the block maximum of the backbone is that of y.  Metadata: the 8-bit
// keep mask of plain 4:8 (whole pairs set).
template <class Q>
__device__ __forceinline__ void backbone_48p(const float (&y)[32], const Q& qz, uint32_t (&codes)[2],
                                             uint32_t& meta, float (&R)[32]) {
  codes[0] = codes[1] = 0u;
  meta = 0u;
  // groups from the last to the first: the metadata is shifted in from its
  // top bit down
#pragma unroll
  for (int g = 3; g >= 0; --g) {
    const float* e = y + 8 * g;
    const float s0 = fmaxf(fabsf(e[0]), fabsf(e[1])), s1 = fmaxf(fabsf(e[2]), fabsf(e[3]));
    const float s2 = fmaxf(fabsf(e[4]), fabsf(e[5])), s3 = fmaxf(fabsf(e[6]), fabsf(e[7]));
    lmask p0, p1, p2, p3;
    top2of4(s0, s1, s2, s3, p0, p1, p2, p3);
    // first kept pair (a) and second (b), ascending K
    const float a0 = lsel(p0, e[0], lsel(p1, e[2], e[4])), a1 = lsel(p0, e[1], lsel(p1, e[3], e[5]));
    const float b0 = lsel(p3, e[6], lsel(p2, e[4], e[2])), b1 = lsel(p3, e[7], lsel(p2, e[5], e[3]));
    meta = push_bit(meta, p3);
    meta = push_bit(meta, p3);
    meta = push_bit(meta, p2);
    meta = push_bit(meta, p2);
    meta = push_bit(meta, p1);
    meta = push_bit(meta, p1);
    meta = push_bit(meta, p0);
    meta = push_bit(meta, p0);
    // the group's four codes go to bytes 2 g (pair a) and 2 g + 1 (pair b)
    put_pair_dyn(qz, codes[g >> 1], 2 * g, a0, a1);
    put_pair_dyn(qz, codes[g >> 1], 2 * g + 1, b0, b1);
    const v2f da = get_pair_dyn(qz, codes[g >> 1], 2 * g);
    const v2f db = get_pair_dyn(qz, codes[g >> 1], 2 * g + 1);
    const float ra0 = a0 - da.x, ra1 = a1 - da.y, rb0 = b0 - db.x, rb1 = b1 - db.y;
    R[8 * g + 0] = lsel(p0, ra0, e[0]);
    R[8 * g + 1] = lsel(p0, ra1, e[1]);
    R[8 * g + 2] = lsel(p1, lsel(p0, rb0, ra0), e[2]);
    R[8 * g + 3] = lsel(p1, lsel(p0, rb1, ra1), e[3]);
    R[8 * g + 4] = lsel(p2, lsel(p3, ra0, rb0), e[4]);
    R[8 * g + 5] = lsel(p2, lsel(p3, ra1, rb1), e[5]);
    R[8 * g + 6] = lsel(p3, rb0, e[6]);
    R[8 * g + 7] = lsel(p3, rb1, e[7]);
  }
}

__device__ __forceinline__ float absmax32(const float* v) {
  float m = 0.0f;
#pragma unroll
  for (int k = 0; k < 32; ++k) m = fmaxf(m, fabsf(v[k]));
  return m;
}

__device__ __forceinline__ float absmax16(const float* v) {
  float m = 0.0f;
#pragma unroll
  for (int k = 0; k < 16; ++k) m = fmaxf(m, fabsf(v[k]));
  return m;
}

// Where one block's outputs go.  spc / spm may be NULL when the dense
// backbone copy spd is given (the compressed backbone is then not written);
// dbg_mask (optional): the block's 32 keep bits.
struct BlockOut {
  uint8_t *spc, *spm, *sps, *dnc, *dns, *spd;
  uint32_t* dbg_mask;
};

// Quantize and store one MXFP4 block: backbone + residual.  The group maximum
// is always kept, so the backbone block max equals the block max of y.
// d.spd (optional): the backbone's dense codes (16 bytes, dropped positions
// 0), the GEMM-ready copy that spares the GEMM the expansion; without d.spc
// only that copy is written.  rule_bias: the E8M0 rule (kE8Floor, kE8Ceil).
template <int PAT>
__device__ __forceinline__ void block_mx(const float (&y)[32], const BlockOut& d, uint32_t rule_bias) {
  const int e = mx_exponent(__float_as_uint(absmax32(y)), rule_bias);
  const MxQ qb = MxQ::make(e);
  uint32_t codes[2] = {0u, 0u}, meta = 0u;
  float R[32];
  if (PAT == 24 && d.spd != nullptr && d.spc == nullptr && d.dbg_mask == nullptr) {
    uint32_t dense[4];
    backbone_24_dense_only(y, qb, dense, R);
    *reinterpret_cast<uint4*>(d.spd) = make_uint4(dense[0], dense[1], dense[2], dense[3]);
  } else if (PAT == 24 && d.spd != nullptr) {
    uint32_t dense[4];
    backbone_24_dense(y, qb, codes, meta, dense, R);
    *reinterpret_cast<uint4*>(d.spd) = make_uint4(dense[0], dense[1], dense[2], dense[3]);
  } else if (PAT == 24) {
    backbone_24(y, qb, codes, meta, R);
  } else if (d.spd != nullptr && d.spc == nullptr && d.dbg_mask == nullptr) {   // 4:8, dense copy alone
    uint32_t dense[4];
    if (PAT == 49) backbone_48p_dense_only(y, qb, dense, R);
    else backbone_48_dense_only(y, qb, dense, R);
    *reinterpret_cast<uint4*>(d.spd) = make_uint4(dense[0], dense[1], dense[2], dense[3]);
  } else if (PAT == 49) {
    backbone_48p(y, qb, codes, meta, R);
  } else {
    backbone_48(y, qb, codes, meta, R);
  }
  const int er = mx_exponent(__float_as_uint(absmax32(R)), rule_bias);
  const MxQ qr = MxQ::make(er);
  uint32_t dn[4];
#pragma unroll
  for (int w = 0; w < 4; ++w) dn[w] = enc8(R + 8 * w, qr);
  if (d.spc != nullptr) {
    *reinterpret_cast<uint2*>(d.spc) = make_uint2(codes[0], codes[1]);
    *reinterpret_cast<uint32_t*>(d.spm) = meta;
  }
  *d.sps = (uint8_t)(e + 127);
  *reinterpret_cast<uint4*>(d.dnc) = make_uint4(dn[0], dn[1], dn[2], dn[3]);
  *d.dns = (uint8_t)(er + 127);
  if (PAT != 24 && d.spd != nullptr && (d.spc != nullptr || d.dbg_mask != nullptr))
    *reinterpret_cast<uint4*>(d.spd) = expand_block<48>(make_uint2(codes[0], codes[1]), meta);
  if (d.dbg_mask) *d.dbg_mask = keep_bits<PAT>(meta);
}

// Quantize and store one NVFP4 block: E4M3 backbone scale per 32 positions,
// E4M3 residual scales per 16 positions (two bytes), per-tensor scale S.
// d.spd (optional): the backbone's dense codes, as in block_mx; without d.spc
// only that copy is written.  Unlike block_mx, the dense copy is always
// expanded from the compressed codes: an NVFP4 code costs a correctly rounded
// division, so converting only the kept values and moving nibbles is cheaper
// than converting every position with zeros at the dropped ones.
template <int PAT>
__device__ __forceinline__ void block_nv(const float (&y)[32], float S, float six_s, const BlockOut& d) {
  const NvQ qb = NvQ::make(absmax32(y), six_s, S);
  uint32_t codes[2], meta;
  float R[32];
  if (PAT == 24)
    backbone_24(y, qb, codes, meta, R);
  else if (PAT == 49)
    backbone_48p(y, qb, codes, meta, R);
  else
    backbone_48(y, qb, codes, meta, R);
  const NvQ q0 = NvQ::make(absmax16(R), six_s, S);
  const NvQ q1 = NvQ::make(absmax16(R + 16), six_s, S);
  const uint32_t dn0 = enc8(R, q0), dn1 = enc8(R + 8, q0), dn2 = enc8(R + 16, q1), dn3 = enc8(R + 24, q1);
  if (d.spc != nullptr) {
    *reinterpret_cast<uint2*>(d.spc) = make_uint2(codes[0], codes[1]);
    *reinterpret_cast<uint32_t*>(d.spm) = meta;
  }
  *d.sps = (uint8_t)e4m3_bits(qb.d);
  *reinterpret_cast<uint4*>(d.dnc) = make_uint4(dn0, dn1, dn2, dn3);
  d.dns[0] = (uint8_t)e4m3_bits(q0.d);
  d.dns[1] = (uint8_t)e4m3_bits(q1.d);
  if (d.spd != nullptr)
    *reinterpret_cast<uint4*>(d.spd) = expand_block<PAT == 24 ? 24 : 48>(make_uint2(codes[0], codes[1]), meta);
  if (d.dbg_mask) *d.dbg_mask = keep_bits<PAT == 49 ? 48 : PAT>(meta);
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

// Cross-lane exchanges on the VALU, no LDS.  Each stage adds the partner
// group of lanes that an xor butterfly over lane masks 1, 2, 4, 8, 16, 32
// would add: DPP quad permutes for 1 and 2; once the lanes of a quad (then of
// a half row) agree, the row half-mirror and row mirror read a lane of the
// partner quad (half row); gfx950's permlane16 / permlane32 swaps exchange
// the rows of 16 and the halves of 32.  fp32 addition is commutative, so
// every lane ends with the same balanced-tree sum as the butterfly.
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

template <class Op>
__device__ __forceinline__ float wave_reduce(float v, Op op) {
  v = op(v, dpp_f32<0xB1>(v));    // quad_perm [1, 0, 3, 2]: lane ^ 1
  v = op(v, dpp_f32<0x4E>(v));    // quad_perm [2, 3, 0, 1]: lane ^ 2
  v = op(v, dpp_f32<0x141>(v));   // row_half_mirror: the other quad of 8
  v = op(v, dpp_f32<0x140>(v));   // row_mirror: the other half of 16
  {
    const auto p = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = op(__uint_as_float(p[0]), __uint_as_float(p[1]));   // rows 2i and 2i + 1
  }
  {
    const auto p = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = op(__uint_as_float(p[0]), __uint_as_float(p[1]));   // lanes 0-31 and 32-63
  }
  return v;
}

__device__ __forceinline__ float wave_tree_sum(float v) {
  return wave_reduce(v, [](float a, float b) { return a + b; });
}

// Output addressing.  Every buffer is panel-major: K is cut into panels of
// 128 positions (4 scale blocks; the last panel may be narrower) and panel p
// stores the bytes of all M rows for its K range, row after row.  Block b of
// a row is block j = b % 4 of panel p = b / 4.  The NVFP4 residual keeps two
// scale bytes per block (blocks of 16).
struct ActOut {
  uint8_t *spc, *spm, *sps, *dnc, *dns;
  int64_t M;
  int K;
  uint8_t* spd;          // MXFP4: the dense backbone copy, or NULL (spc / spm may then be NULL)
  uint32_t rule_bias;    // MXFP4: E8M0 rule (kE8Floor or kE8Ceil)
  uint32_t* dbg_mask;    // optional: 32 keep bits per block, laid out like the 4:8 metadata
  float* dbg_r;          // optional: the RMSNorm reciprocal r of every row
};

// Panel-major order is block-major order: block b of a row is block number
// V = 4 M p + row (wp / 32) + j (p = b / 4, j = b % 4, wp = panel width), and
// every buffer holds its bytes for block V at V times its bytes per block.
__device__ __forceinline__ int64_t block_index(int64_t M, int K, int64_t row, int b) {
  const int p = b >> 2, j = b & 3;
  const int wp = min(128, K - 128 * p);
  return (int64_t)p * M * 4 + row * (wp / 32) + j;
}

template <bool NV>
__device__ __forceinline__ BlockOut block_at(const ActOut& o, int64_t V) {
  BlockOut r;
  r.dnc = o.dnc + V * 16;
  r.spc = o.spc ? o.spc + V * 8 : nullptr;
  r.spm = o.spm ? o.spm + V * 4 : nullptr;
  r.sps = o.sps + V;
  r.dns = o.dns + (NV ? V * 2 : V);
  r.spd = o.spd ? o.spd + V * 16 : nullptr;
  r.dbg_mask = o.dbg_mask ? o.dbg_mask + V : nullptr;
  return r;
}

template <bool NV>
__device__ __forceinline__ BlockOut block_out(const ActOut& o, int64_t row, int b) {
  return block_at<NV>(o, block_index(o.M, o.K, row, b));
}

template <int PAT, bool NV>
__device__ __forceinline__ void block_out_write(const float (&y)[32], const ActOut& o, int64_t row, int b, float S,
                                                float six_s) {
  const BlockOut d = block_out<NV>(o, row, b);
  if (NV) {
    block_nv<PAT>(y, S, six_s, d);
  } else {
    block_mx<PAT>(y, d, o.rule_bias);
  }
}

__device__ __forceinline__ float wave_max(float v) {
  return wave_reduce(v, [](float a, float b) { return fmaxf(a, b); });
}

// The activation rows a preparation reads.  Without a residual input they
// are X itself.  With one -- the residual add that precedes a transformer
// block's RMSNorm, fused into the preparation on the producer side -- a row
// is h = bf16(x + res): the two bf16 values added in fp32 and rounded to
// nearest even once.  The preparation kernels also write h to H (the updated
// residual stream, which may be the residual input itself) and then work on
// h; the NVFP4 amax pre-pass recomputes h without writing it.
struct XSrc {
  const uint16_t* X;
  int64_t ldx;
  const uint16_t* Rs;
  int64_t ldr;
  uint16_t* H;
  int64_t ldh;
};

__device__ __forceinline__ uint32_t add_bf16x2(uint32_t a, uint32_t b) {
  typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
  bf2 v;
  v[0] = (__bf16)(bf16_lo(a) + bf16_lo(b));   // v_cvt_pk_bf16_f32: nearest even
  v[1] = (__bf16)(bf16_hi(a) + bf16_hi(b));
  return __builtin_bit_cast(uint32_t, v);
}

// e^x for x <= 0 in fp32, every step an IEEE fp32 operation rounded to
// nearest even (the file is compiled without contraction): Cody-Waite
// argument reduction (Cody and Waite, "Software Manual for the Elementary
// Functions", 1980) x = k ln2 + r, k = rint(x log2 e), with ln2 split into a
// 16-bit head (k * head exact for |k| < 2^8) and an fp32 tail; the degree-7
// Taylor polynomial of e^r in Horner form; then one multiply by the exact
// power of two 2^k, which rounds into the subnormal range below 2^-126.
// Results below 2^-149 are 0.  Within 2 ulp of e^x.
__device__ __forceinline__ float exp_nonpositive(float x) {
  const float k = __builtin_rintf(x * 0x1.715476p+0f);
  const float r = (x - k * 0x1.62e4p-1f) - k * 0x1.7f7d1cp-20f;
  float p = 0x1.a01a02p-13f;        // 1/7!
  p = p * r + 0x1.6c16c2p-10f;      // 1/6!
  p = p * r + 0x1.111112p-7f;       // 1/5!
  p = p * r + 0x1.555556p-5f;       // 1/4!
  p = p * r + 0x1.555556p-3f;       // 1/3!
  p = p * r + 0.5f;
  p = p * r + 1.0f;
  p = p * r + 1.0f;
  const int ki = (int)k;
  return ki < -149 ? 0.0f : p * exp2_int(ki);
}

// SiLU(g) * u in fp32 for the down projection's input (the SiLU.mul that
// follows the gate/up projection, fused into the preparation on the producer
// side): t = e^-|g|, q = 1 + t, s = g / q (g >= 0) or (g t) / q (g < 0) --
// SiLU(g) = g / (1 + e^-g) = g e^g / (1 + e^g) -- with correctly rounded
// division, then s u.  One fixed fp32 recipe, so h = bf16(s u) is a
// deterministic function of (g, u), within one bf16 step of the exactly
// rounded SiLU(g) u.
__device__ __forceinline__ float silu_mul(float g, float u) {
  const float t = exp_nonpositive(-fabsf(g));
  const float q = 1.0f + t;
  const float num = g >= 0.0f ? g : g * t;
  return (num / q) * u;
}

__device__ __forceinline__ uint32_t silu_mul_bf16x2(uint32_t g, uint32_t u) {
  typedef __bf16 bf2 __attribute__((ext_vector_type(2)));
  bf2 v;
  v[0] = (__bf16)silu_mul(bf16_lo(g), bf16_lo(u));   // nearest even
  v[1] = (__bf16)silu_mul(bf16_hi(g), bf16_hi(u));
  return __builtin_bit_cast(uint32_t, v);
}

// Sources of the rows a preparation reads (SRC): 0, X itself; 1, the residual
// add h = bf16(x + res) (Rs = res); 2, SiLU.mul h = bf16(SiLU(g) * u) (X = g,
// Rs = u).  Block b (32 values, four 16-byte pieces) of `row` is loaded and h
// formed; when write_h (and, for SiLU.mul, H given) it is stored.  Every
// (row, block) is stored by exactly one lane, which read its inputs before:
// in place is safe.
template <int SRC>
__device__ __forceinline__ void load_block(const XSrc& s, int64_t row, int b, uint4 (&q)[4], bool write_h) {
  const uint4* xr = reinterpret_cast<const uint4*>(s.X + row * s.ldx);
#pragma unroll
  for (int j = 0; j < 4; ++j) q[j] = xr[4 * b + j];
  if (SRC != 0) {
    const uint4* rr = reinterpret_cast<const uint4*>(s.Rs + row * s.ldr);
    uint4 rq[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) rq[j] = rr[4 * b + j];
    if (SRC == 1) {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        q[j] = make_uint4(add_bf16x2(q[j].x, rq[j].x), add_bf16x2(q[j].y, rq[j].y), add_bf16x2(q[j].z, rq[j].z),
                          add_bf16x2(q[j].w, rq[j].w));
    } else {
#pragma unroll
      for (int j = 0; j < 4; ++j)
        q[j] = make_uint4(silu_mul_bf16x2(q[j].x, rq[j].x), silu_mul_bf16x2(q[j].y, rq[j].y),
                          silu_mul_bf16x2(q[j].z, rq[j].z), silu_mul_bf16x2(q[j].w, rq[j].w));
    }
    if (write_h && (SRC == 1 || s.H != nullptr)) {
      uint4* hr = reinterpret_cast<uint4*>(s.H + row * s.ldh);
#pragma unroll
      for (int j = 0; j < 4; ++j) hr[4 * b + j] = q[j];
    }
  }
}

// Load a row's blocks (NB per lane) and return its RMSNorm reciprocal r.
template <int NB, bool RES>
__device__ __forceinline__ float load_row_rms(const XSrc& src, int64_t row, bool write_h, int lane, int nblk, int K,
                                              float eps, uint4 (&xs)[NB][4]) {
  float chunk[NB];
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int b = lane + 64 * i;
    if (b < nblk) {
      load_block<RES>(src, row, b, xs[i], write_h);
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
  return (float)(1.0 / __builtin_sqrt((double)chunk[0] / (double)K + (double)eps));
}

// y = (x * r) * gamma for one block (gq: the block's 32 bf16 gamma values).
__device__ __forceinline__ void norm_block(const uint4 (&xq)[4], const uint4 (&gq)[4], float r, float (&y)[32]) {
  float x[32], g[32];
  unpack_bf16x32(xq, x);
  unpack_bf16x32(gq, g);
#pragma unroll
  for (int k = 0; k < 32; ++k) {
    const float t = x[k] * r;
    y[k] = t * g[k];
  }
}

}  // namespace sharq
