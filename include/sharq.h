/*
 * sharq.h -- C ABI of the SharQ sparse-dense FP4 linear layer for AMD Instinct
 * MI355X (gfx950).
 *
 * SharQ (arXiv 2606.26587) approximates a linear layer Y = X W^T by splitting
 * the activation online into an N:M sparse FP4 backbone and a dense FP4
 * residual taken against the *dequantized* backbone, then summing two FP4
 * GEMMs that read one shared FP4 weight payload (Sec. 3.3 eqs.
 * "sharq-sparse-backbone", "sharq-quantized-backbone", "sharq-residual",
 * "sharq-output"; Sec. 3.4).
 *
 * Conventions for every entry point
 *   - Tensor pointers are DEVICE pointers owned by the caller; the library
 *     allocates nothing, keeps no global state and never synchronizes.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream);
 *     all work is enqueued asynchronously on it.
 *   - Errors are returned, never thrown.  Arguments are validated before any
 *     launch: SHARQ_EINVAL (NULL pointer, negative size, K not a positive
 *     multiple of 32, K % m != 0, leading dimension < K or < N),
 *     SHARQ_EUNSUPPORTED (a format / pattern / dtype combination that is not
 *     built), SHARQ_EALIGN (a pointer not aligned as stated below),
 *     SHARQ_EHIP (the HIP runtime reported an error at launch).
 *   - Inputs must be finite; NaN or Inf inputs give unspecified results.
 *   - Row counts of 0 are valid and launch nothing; the buffers of an empty
 *     tensor may then be NULL.
 *
 * Numeric formats (App. A.1 of the paper)
 *   E2M1 element code: bit 3 = sign, bits 0-2 index {0, .5, 1, 1.5, 2, 3, 4, 6}.
 *   MXFP4: E2M1 + one E8M0 scale per 32 consecutive K values; E8M0 code c
 *          means 2^(c-127).  NVFP4: E2M1 + one E4M3 scale (bias 7, max 448)
 *          per block + one fp32 per-tensor scale.
 *   HiF4 (App. "HiFloat4 (HiF4) Data Format"): units of 64 K positions; each
 *          element an S1P2 code (bit 3 sign, bits 0-2 magnitude m, value
 *          m/4); per unit 4 metadata bytes [E6M2, E1_8, E1_16 low, E1_16
 *          high]: an E6M2 scale (6 exponent bits, bias 48, 2 mantissa bits,
 *          normal values only) and one-bit micro-exponents per 8 and per 4
 *          elements (bit j = group j); value = E6M2 * 2^(E1_8 + E1_16) *
 *          S1P2 (eq. "hif4-value").  The 4 bytes of a unit occupy the 2-byte
 *          scale slots of its two 32-position blocks.  K must be a multiple of
 *          64; built with the 2:4 pattern, SHARQ_MODE_SHARQ, no grouped form.
 *   Two 4-bit codes per byte, the element with the lower K index in the low
 *   nibble.
 *
 * Buffer layout: PANEL-MAJOR.  Every buffer below holds a fixed number of
 * bytes per 32 consecutive K positions of a row (its "row bytes").  K is cut
 * into panels of SHARQ_PANEL_K = 128 positions (the last panel is narrower
 * when K % 128 != 0); panel p stores the row bytes of ALL rows of the tensor
 * for K range [128 p, 128 p + width_p), row after row, and panels follow each
 * other.  Byte offset of (panel p, row r) in a buffer with b bytes per 32 K
 * positions and R rows: p * R * 4 b + r * (width_p / 32) * b.  A tile of
 * consecutive rows is thus one contiguous run per panel, which is how the
 * GEMM streams it; a single row is still addressable (row gathers).  The
 * total size equals the row-major size R * (K / 32) * b.
 */
#ifndef SHARQ_H
#define SHARQ_H

#define SHARQ_PANEL_K 128

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#ifndef SHARQ_API
#define SHARQ_API __attribute__((visibility("default")))
#endif

typedef enum {
  SHARQ_OK = 0,
  SHARQ_EINVAL = 1,
  SHARQ_EUNSUPPORTED = 2,
  SHARQ_EALIGN = 3,
  SHARQ_EHIP = 4
} sharq_status;

typedef enum { SHARQ_MXFP4 = 0, SHARQ_NVFP4 = 1, SHARQ_HIF4 = 2 } sharq_format;

typedef enum { SHARQ_BF16 = 0, SHARQ_F16 = 1, SHARQ_F32 = 2 } sharq_dtype;

/* N:M activation pattern: keep the n largest magnitudes of every m consecutive
 * K positions (eq. "dynamic-mask").  pairs = 1 selects in pairs, NVFP4's
 * "4:8 in pairs" (App. A.1.4; Fig. 2 "pair-topk"): the m positions of a group
 * are m/2 adjacent pairs (2i, 2i+1), and the n/2 pairs with the largest score
 * max(|y_2i|, |y_2i+1|) survive whole (ties -> lower pair).  Built: 2:4, 4:8
 * and 4:8 in pairs (with either format). */
typedef struct {
  int32_t n, m;
  int32_t pairs;   /* 0: element-wise top-n, 1: in pairs */
} sharq_pattern;

/*
 * E8M0 scale rule of MXFP4 (ablation flag).  SHARQ_SCALE_FLOOR, the default,
 * is the OCP Microscaling rule e = floor(log2 amax) - 2: a block peak above
 * 6 * 2^e saturates at 6.  SHARQ_SCALE_CEIL takes e = ceil(log2(amax / 6)),
 * the group scale amax / 6 of Sec. 3.1 eq. "group-quant" rounded up to a
 * power of two so that nothing clips (App. A.1.1: a power-of-two scale cannot
 * bring every block peak to the E2M1 maximum).  Both clamp at -127 and give
 * -127 to an all-zero block.  Built for MXFP4 in SHARQ_MODE_SHARQ.
 */
typedef enum { SHARQ_SCALE_FLOOR = 0, SHARQ_SCALE_CEIL = 1 } sharq_scale_rule;

/*
 * Path combination of a prepared activation (Sec. 4.4, table
 * "ablation-combination"; Sec. 3.1 eq. "direct-sparse-quant"; the
 * round-to-nearest FP4 rows of table "ablation-format").  Every mode has two
 * path slots: path 1 quantizes y, path 2 quantizes the residual of y against
 * path 1's dequantized values; the GEMM sums the paths' products into one
 * accumulator.  A sparse path keeps the top n of every m of ITS OWN input and
 * quantizes the kept values in blocks of 32 logical positions (the backbone
 * quantizer); a dense path is the format's plain quantizer (MXFP4 per 32,
 * NVFP4 per 16).  NVFP4 uses one per-tensor scale for both paths.
 *
 *   mode                       path 1   path 2
 *   SHARQ_MODE_SHARQ           sparse   dense     the method (default, 0)
 *   SHARQ_MODE_SPARSE          sparse   -         no residual compensation
 *   SHARQ_MODE_DENSE           -        dense     plain FP4 (RTN), i.e. n = 0
 *   SHARQ_MODE_DENSE_DENSE     dense    dense     two dense paths
 *   SHARQ_MODE_SPARSE_SPARSE   sparse   sparse    second mask chosen on |R|
 *
 * Only SHARQ_MODE_SHARQ is the method; the others exist for ablation.  They
 * run on generic (non-interleaved) GEMM kernels and are not built for the
 * grouped form or with the fused residual add.
 */
typedef enum {
  SHARQ_MODE_SHARQ = 0,
  SHARQ_MODE_SPARSE = 1,
  SHARQ_MODE_DENSE = 2,
  SHARQ_MODE_DENSE_DENSE = 3,
  SHARQ_MODE_SPARSE_SPARSE = 4
} sharq_mode;

/*
 * A prepared activation: the output of sharq_prepare, the input of
 * sharq_linear / sharq_linear_grouped.  One row per token; panel-major (see
 * above).  Row bytes per row are listed as [rows][...].  In SHARQ_MODE_SHARQ:
 *
 *   sp_codes [rows][K*n/m/2]  backbone E2M1 codes of the kept positions only,
 *                             in ascending K order (Sec. 3.4: "quantizes and
 *                             compresses it"); 16-byte aligned.
 *   sp_meta  [rows][K/8]      which positions were kept.  2:4: per group of 4
 *                             the two kept indices i0 < i1 as i0 | i1 << 2 (a
 *                             nibble), two groups per byte, even group low.
 *                             4:8 (also in pairs): per group of 8 an 8-bit
 *                             keep mask (bit p = position p kept).  4-byte
 *                             aligned.
 *   sp_scale [rows][K/32]     backbone block scale per 32 logical K positions
 *                             (Fig. 2 "sparse group-32 scales"): E8M0 (MXFP4)
 *                             or E4M3 (NVFP4); HiF4: [rows][K/16], the unit
 *                             metadata of each 64 logical positions.
 *   dn_codes [rows][K/2]      residual E2M1 codes, all positions; 16-byte aligned.
 *   dn_scale [rows][K/32] (MXFP4, E8M0) | [rows][K/16] (NVFP4, E4M3; HiF4,
 *                             unit metadata).
 *   tensor_scale              NVFP4: one fp32 per-tensor scale S (device); the
 *                             element value is code * block_scale * S.
 *                             MXFP4: unused (may be NULL).
 *   mode                      SHARQ_MODE_SHARQ (0).
 *   dn_meta                   unused (may be NULL).
 *   sp_dense [rows][K/2]      optional (NULL = none), MXFP4 and NVFP4 (not
 *                             HiF4): the backbone's codes at all K positions
 *                             (dropped positions code 0), laid out like
 *                             dn_codes, with the backbone's scales sp_scale;
 *                             16-byte aligned.  When given, the preparation
 *                             writes it beside the compressed form, and the
 *                             main kernels of sharq_linear and (MXFP4)
 *                             sharq_linear_grouped (K a multiple of 128) read
 *                             it instead of expanding sp_codes / sp_meta:
 *                             gfx950 has no sparse FP4 matrix instruction, so
 *                             the backbone runs dense anyway, and the copy
 *                             (K/2 more bytes per row) takes the expansion
 *                             out of every column tile.
 *                             Dense-only form: with sp_dense given, sp_codes
 *                             and sp_meta may both be NULL (K a multiple of
 *                             128, SHARQ_MODE_SHARQ); the preparation then
 *                             writes the backbone as the dense copy alone
 *                             (0.5 B per element instead of 0.375 + 0.5), and
 *                             every GEMM reads that copy.
 *   scale_rule                sharq_scale_rule of both paths' E8M0 scales
 *                             (MXFP4; SHARQ_SCALE_FLOOR = 0 by default).
 *   dbg_mask [rows][K/8]      optional (NULL = none) debug output of
 *                             sharq_prepare: the N:M keep mask, bit p of every
 *                             group of 8 positions set when position p was
 *                             kept, laid out like the 4:8 metadata (4 bytes
 *                             per 32 positions, panel-major); 4-byte aligned.
 *   dbg_r    [rows] fp32      optional debug output: the RMSNorm reciprocal r
 *                             of every row (written only when gamma is given).
 *                             Both are for parity triage; MXFP4 and NVFP4,
 *                             SHARQ_MODE_SHARQ.
 *
 * Other modes: path 1 lives in sp_codes / sp_meta / sp_scale and path 2 in
 * dn_codes / dn_meta / dn_scale.  A sparse path has the backbone layout above
 * (codes [rows][K*n/m/2], meta [rows][K/8], scale [rows][K/32]); a dense path
 * the residual layout (codes [rows][K/2], no meta, scale [rows][K/32] MXFP4 or
 * [rows][K/16] NVFP4); an absent path's buffers are unused and may be NULL.
 * sharq_act_buffer_bytes_mode gives every size (0 = unused).  Alignment as
 * above (dn_meta 4-byte aligned).
 */
typedef struct {
  int64_t rows, K;
  sharq_format fmt;
  sharq_pattern nm;
  uint8_t *sp_codes;
  uint8_t *sp_meta;
  uint8_t *sp_scale;
  uint8_t *dn_codes;
  uint8_t *dn_scale;
  float *tensor_scale;
  sharq_mode mode;
  uint8_t *dn_meta;
  uint8_t *sp_dense;
  sharq_scale_rule scale_rule;
  uint8_t *dbg_mask;
  float *dbg_r;
} sharq_act;

/*
 * A quantized weight: ONE shared FP4 payload for both paths with
 * path-specific scale views (Sec. 3.4 "Shared FP4 weights with path-specific
 * scales"; Fig. 2).  W is [N][K] (out-features x in-features), Y = X W^T;
 * each expert's buffers are panel-major over its N rows.
 * `experts` weights of identical shape may be stacked back to back (MoE);
 * expert e starts at codes + e*N*K/2 and scale + e*N*(K/32).
 *
 *   codes    [experts][N][K/2]   E2M1, 16-byte aligned.
 *   scale    [experts][N][K/32]  E8M0 (MXFP4, both paths) or E4M3 (NVFP4,
 *                                sparse view: one scale per 32).
 *   scale_dn [experts][N][K/16]  NVFP4 dense view: each per-32 scale repeated
 *                                for its two 16-element halves.  MXFP4: equal
 *                                to `scale`.
 *   HiF4: scale [experts][N][K/16] holds the unit metadata, one view for
 *   both paths (scale_dn unused, may equal `scale`).
 *   tensor_scale [experts]       NVFP4 per-tensor scale(s) S_w (device);
 *                                MXFP4: unused.
 *   scale_rule                   MXFP4: the sharq_scale_rule sharq_quantize_weight
 *                                applies (the GEMMs ignore it).
 */
typedef struct {
  int64_t N, K, experts;
  sharq_format fmt;
  uint8_t *codes;
  uint8_t *scale;
  uint8_t *scale_dn;
  float *tensor_scale;
  sharq_scale_rule scale_rule;
} sharq_weight;

/* Bytes of each buffer of a prepared activation / quantized weight (host-side
 * sizing helpers, no device work).  Return 0 for an invalid combination. */
SHARQ_API size_t sharq_act_buffer_bytes(int64_t rows, int64_t K, sharq_format fmt, sharq_pattern nm,
                              int32_t which /* 0 sp_codes, 1 sp_meta, 2 sp_scale, 3 dn_codes, 4 dn_scale */);
SHARQ_API size_t sharq_weight_buffer_bytes(int64_t N, int64_t K, sharq_format fmt,
                                 int32_t which /* 0 codes, 1 scale, 2 scale_dn */);
/* Buffer sizes of a prepared activation in a given mode; which 5 = dn_meta.
 * 0 for a buffer the mode does not use, or for an invalid combination. */
SHARQ_API size_t sharq_act_buffer_bytes_mode(int64_t rows, int64_t K, sharq_format fmt, sharq_pattern nm,
                                   sharq_mode mode, int32_t which);

/*
 * Quantize a weight W [N][K] (row stride ldw elements, dtype wdt = BF16 or
 * F32) once into the shared FP4 payload and its scale views (Fig. 2 "weight
 * preparation").  MXFP4: per row, per 32 K values, E8M0 = floor(log2 amax) - 2
 * (OCP rule, clamped at -127), codes = E2M1(w / 2^e), ties to even, saturating.
 * (out->scale_rule = SHARQ_SCALE_CEIL: ceil(log2(amax / 6)) instead).
 * NVFP4: S_w = amax(W)/2688 computed on the device, E4M3 per 32, dense view
 * duplicated per 16.  HiF4: units of 64 along K, the conversion of the HiF4
 * appendix (its algorithm "bf16-to-hif4") on the fp32 values.  `out` fields
 * N, K, fmt, scale_rule and the buffers must be set by the caller; experts
 * must be 1.  The format and the rule travel in `out` rather than as
 * arguments, so that the weight descriptor records what its bytes mean.
 */
SHARQ_API sharq_status sharq_quantize_weight(const void *W, sharq_dtype wdt, int64_t N, int64_t K, int64_t ldw,
                                   sharq_weight *out, void *stream);

/*
 * Fused activation preparation (Sec. 3.4 "Fused sparse-residual preparation";
 * Fig. 2): one kernel that, per row of X [M][K] (row stride ldx elements,
 * dtype xdt = BF16):
 *   1. if gamma != NULL (bf16 [K]): y = (x * r) * gamma with
 *      r = 1/sqrt(mean(x^2) + eps) (sum of squares as a balanced binary tree
 *      in fp32, r rounded from fp64); else y = x;
 *   2. keeps the n largest |y| of every group of m (ties -> lower index),
 *      or the n/2 best pairs when nm.pairs = 1;
 *   3. quantizes the kept values per 32 logical positions (backbone);
 *   4. forms the residual R = y - dequant(backbone) (eq. "sharq-residual");
 *   5. quantizes R densely.
 * NVFP4 additionally needs the per-tensor scale S: if tensor_scale_in is NULL
 * the library computes S = amax(y)/2688 over the whole call in a pre-pass
 * (one more read of X) and writes it to out->tensor_scale; otherwise
 * *tensor_scale_in (device) is used and copied there.
 * out->rows, K, fmt, nm and the buffers must match the arguments.
 * out->mode selects the path combination (see sharq_mode): steps 2-5 then
 * become path 1 on y, the residual R = y - dequant(path 1), and path 2 on R.
 * A mode with a sparse path needs a built pattern; SHARQ_MODE_DENSE and
 * SHARQ_MODE_DENSE_DENSE ignore nm (it must still be valid).
 */
SHARQ_API sharq_status sharq_prepare(const void *X, sharq_dtype xdt, int64_t M, int64_t K, int64_t ldx,
                           const void *gamma, float eps, sharq_pattern nm, sharq_format fmt,
                           const float *tensor_scale_in, sharq_act *out, void *stream);

/*
 * Preparation with the residual add that precedes a transformer block's
 * RMSNorm fused in on the producer side (Sec. 4.3: the preparation absorbs
 * the preprocessing steps of the data flow instead of running them as
 * separate operators).  Per element, h = bf16(x + residual): the two bf16
 * values added in fp32 and rounded to nearest even once.  h is written to
 * h_out (bf16 [M][K], row stride ldh; it may be `residual` itself, updated in
 * place, when ldh == ldr) and then prepared exactly as sharq_prepare prepares
 * X.  residual: bf16 [M][K], row stride ldr.  Both 16-byte aligned with
 * 16-byte row strides.  With NVFP4 and no tensor_scale_in the amax pre-pass
 * forms h as well.  Other arguments, errors and outputs as for sharq_prepare;
 * out->mode must be SHARQ_MODE_SHARQ (others: SHARQ_EUNSUPPORTED).
 */
SHARQ_API sharq_status sharq_prepare_residual(const void *X, const void *residual, void *h_out, sharq_dtype xdt,
                                    int64_t M, int64_t K, int64_t ldx, int64_t ldr, int64_t ldh,
                                    const void *gamma, float eps, sharq_pattern nm, sharq_format fmt,
                                    const float *tensor_scale_in, sharq_act *out, void *stream);

/*
 * Preparation of a down projection's input with the SiLU.mul that produces it
 * fused in on the producer side (Sec. 4.3: the preparation absorbs the
 * preprocessing steps of the data flow).  Per element,
 * h = bf16(SiLU(g) * u), SiLU(g) = g / (1 + exp(-g)), by one fixed fp32
 * recipe: t = e^-|g| (Cody-Waite argument reduction and the degree-7 Taylor
 * polynomial, within 2 ulp), s = g / (1 + t) for g >= 0 and g t / (1 + t)
 * below (correctly rounded division), h = bf16(s u) to nearest even.  h is
 * thus a fixed function of (g, u), within one bf16 step of the exactly
 * rounded value; inputs must keep s u finite.  h is prepared without RMSNorm
 * exactly as sharq_prepare prepares X, and written to h_out (bf16 [M][K], row stride ldh) when h_out is not NULL.
 * gate, up: bf16 [M][K], row strides ldg, ldu (e.g. the two halves of a
 * gate/up projection's output, ldg = ldu = 2K); 16-byte aligned with 16-byte
 * row strides.  With NVFP4 and no tensor_scale_in the amax pre-pass forms h
 * as well.  Modes other than SHARQ_MODE_SHARQ and HiF4: SHARQ_EUNSUPPORTED.
 * Other arguments, errors and outputs as for sharq_prepare.
 */
SHARQ_API sharq_status sharq_prepare_silu_mul(const void *gate, const void *up, void *h_out, sharq_dtype xdt,
                                    int64_t M, int64_t K, int64_t ldg, int64_t ldu, int64_t ldh,
                                    sharq_pattern nm, sharq_format fmt, const float *tensor_scale_in,
                                    sharq_act *out, void *stream);

/*
 * Two-path output (eq. "sharq-output"; Sec. 3.4 "Residual path compensation
 * by accumulation"): Y [rows][N] (row stride ldy, dtype ydt) =
 *   dequant(backbone) * dequant_sp(W)^T + dequant(residual) * dequant_dn(W)^T,
 * both products accumulated in one fp32 accumulator and written once.
 * The activation and weight formats must match.  MXFP4 runs on the
 * block-scaled FP4 matrix cores; NVFP4 (whose E4M3 block scales those cannot
 * apply) multiplies the exactly dequantized values q * d on 16-bit matrix
 * cores (fp16 for K a multiple of 128, where every q * d is an exact normal
 * fp16 value; bf16 otherwise) and applies S_x * S_w once to the fp32 sums.  NVFP4 needs a->tensor_scale and
 * w->tensor_scale.  For the other modes of a->mode, Y is the sum over the
 * mode's paths, each against the weight's view of its kind (sparse view for a
 * sparse path, dense view for a dense one).
 */
SHARQ_API sharq_status sharq_linear(const sharq_act *a, const sharq_weight *w, void *Y, sharq_dtype ydt,
                          int64_t ldy, void *stream);

/*
 * Preparation and two-path output in one call (Sec. 4.3: the fused
 * preparation, the shared weight and the accumulating residual path keep the
 * data flow close to a single linear kernel; Sec. 3.4; Sec. 3.3 eq.
 * "sharq-output"): exactly sharq_prepare(X ..., act) followed by
 * sharq_linear(act, w, Y ...), with every argument of both validated before
 * anything is launched.  For a few rows (decode: MXFP4, the method's path
 * combination, K a multiple of 128 up to 16384, M <= 4 when the prepared rows
 * fit in LDS) it runs as ONE kernel: each workgroup of the small-M GEMM
 * prepares the rows in its prologue and workgroup 0 writes them to `act`;
 * the outputs (act's buffers and Y) are bit-identical to the two calls.
 */
SHARQ_API sharq_status sharq_prepare_linear(const void *X, sharq_dtype xdt, int64_t M, int64_t K, int64_t ldx,
                                            const void *gamma, float eps, sharq_pattern nm, sharq_format fmt,
                                            const float *tensor_scale_in, sharq_act *act, const sharq_weight *w,
                                            void *Y, sharq_dtype ydt, int64_t ldy, void *stream);

/*
 * Grouped form for mixture-of-experts layers (the MoE configuration of the
 * paper's evaluation, Sec. 4.1-4.2, Qwen3-30B-A3B): the two-path output of
 * Sec. 3.3 eq. "sharq-output" applied per expert to the rows routed to it.
 * For every expert e and every i in [expert_offsets[e], expert_offsets[e+1]),
 *   Y[i] = SharQ(A[row_index ? row_index[i] : i], W_e).
 * The experts' weights are stacked in one sharq_weight (w->experts of them,
 * one shape) rather than passed as an array of descriptors, so that the
 * kernel reads every expert's payload from one base pointer.
 * expert_offsets: device int32 [w->experts + 1], non-decreasing, first 0,
 * last == total.  row_index: device int32 [total], each in [0, a->rows), or
 * NULL.  Y [total][N] (row stride ldy).  Offsets are read on the device; the
 * host never waits for them.  Built for MXFP4 in SHARQ_MODE_SHARQ; NVFP4 or
 * another mode returns SHARQ_EUNSUPPORTED.
 */
SHARQ_API sharq_status sharq_linear_grouped(const sharq_act *a, const int32_t *row_index,
                                  const int32_t *expert_offsets, int64_t total,
                                  const sharq_weight *w, void *Y, sharq_dtype ydt, int64_t ldy,
                                  void *stream);

SHARQ_API const char *sharq_status_str(sharq_status s);

/* Library version string. */
SHARQ_API const char *sharq_version(void);

#ifdef __cplusplus
}
#endif

#endif /* SHARQ_H */
