/*
 * sharq_ref.h -- plain C oracle of the SharQ sparse-dense FP4 linear layer
 * (SharQ, arXiv 2606.26587), TEST INFRASTRUCTURE ONLY.
 *
 * The host-pointer twin of the library's preparation, weight quantization and
 * two-path GEMM for MXFP4 (2:4 and 4:8 element-wise selection, optional
 * RMSNorm, floor or ceil E8M0 rule) and NVFP4 (the same selections and 4:8 in
 * pairs, dynamic or given per-tensor scale), written as straight scalar loops
 * from the paper's definitions and the readings the NumPy oracle lists (R1-R8,
 * R13).
 * It shares no code with the HIP library or the NumPy oracle: only tests, the
 * package's smoke check and the benchmark's CPU-baseline leg use it.
 *
 * Buffers are ROW-MAJOR host arrays (the method's packed representation, not
 * the library's panel-major storage):
 *   sp_codes [M][K*n/m/2]  kept E2M1 codes in ascending K, low nibble first
 *   sp_meta  [M][K/8]      2:4: per group (i0 | i1 << 2), two groups per byte,
 *                          even group in the low nibble; 4:8: a keep mask byte
 *   sp_scale [M][K/32]     E8M0 of the backbone blocks (32 logical positions)
 *   dn_codes [M][K/2]      residual E2M1 codes, low nibble first
 *   dn_scale [M][K/32]     E8M0 of the residual blocks
 *   keep     [M][K/8]      optional: bit p of byte b = position 8 b + p kept
 *   r        [M]           optional: the RMSNorm reciprocal of every row
 *   w codes  [N][K/2], w scale [N][K/32]
 *   Y        [M][ldy] fp64
 * Status codes: 0 ok, 1 invalid argument, 2 unsupported combination (the
 * library's SHARQ_OK / SHARQ_EINVAL / SHARQ_EUNSUPPORTED meanings).
 */
#ifndef SHARQ_REF_H
#define SHARQ_REF_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int sharq_ref_prepare(const uint16_t *X, int64_t M, int64_t K, int64_t ldx, const uint16_t *gamma, float eps,
                      int n, int m, int scale_rule, uint8_t *sp_codes, uint8_t *sp_meta, uint8_t *sp_scale,
                      uint8_t *dn_codes, uint8_t *dn_scale, float *r, uint8_t *keep);

int sharq_ref_quantize_weight(const uint16_t *W, int64_t N, int64_t K, int64_t ldw, int scale_rule, uint8_t *codes,
                              uint8_t *scale);

int sharq_ref_linear(int64_t M, int64_t K, int n, int m, const uint8_t *sp_codes, const uint8_t *sp_meta,
                     const uint8_t *sp_scale, const uint8_t *dn_codes, const uint8_t *dn_scale, int64_t N,
                     const uint8_t *w_codes, const uint8_t *w_scale, double *Y, int64_t ldy);

/*
 * NVFP4 (App. A.1.2-A.1.3, reading R7): the same row-major buffers with E4M3
 * block scales and one fp32 per-tensor scale S, element value
 * code * block scale * S.
 *   sharq_ref_prepare_nv: sp_scale [M][K/32] (backbone blocks of 32 logical
 *     positions), dn_scale [M][K/16] (residual blocks of 16); S from
 *     *tensor_scale_in when given, else fl32(amax(y) / 2688) over the call
 *     (1 when y is all zero), written to *tensor_scale_out.  pairs = 1: 4:8
 *     in pairs (n = 4, m = 8 only).
 *   sharq_ref_quantize_weight_nv: scale [N][K/32], S_w to *tensor_scale; the
 *     weight's dense view repeats each scale over its two 16-position halves.
 *   sharq_ref_linear_nv: Y in fp64 with S_x and S_w applied.
 *   sharq_ref_e4m3_code: the E4M3 code nearest to a >= 0 (ties to the even
 *     code, 448 for anything larger), by exhaustive search.
 */
int sharq_ref_prepare_nv(const uint16_t *X, int64_t M, int64_t K, int64_t ldx, const uint16_t *gamma, float eps,
                         int n, int m, int pairs, const float *tensor_scale_in, float *tensor_scale_out,
                         uint8_t *sp_codes, uint8_t *sp_meta, uint8_t *sp_scale, uint8_t *dn_codes,
                         uint8_t *dn_scale);

int sharq_ref_quantize_weight_nv(const uint16_t *W, int64_t N, int64_t K, int64_t ldw, uint8_t *codes,
                                 uint8_t *scale, float *tensor_scale);

int sharq_ref_linear_nv(int64_t M, int64_t K, int n, int m, const uint8_t *sp_codes, const uint8_t *sp_meta,
                        const uint8_t *sp_scale, const uint8_t *dn_codes, const uint8_t *dn_scale,
                        float tensor_scale_x, int64_t N, const uint8_t *w_codes, const uint8_t *w_scale,
                        float tensor_scale_w, double *Y, int64_t ldy);

uint8_t sharq_ref_e4m3_code(float a);

/* OpenMP threads used over rows (0 or negative: the runtime's default). */
void sharq_ref_set_threads(int threads);
int sharq_ref_max_threads(void);

#ifdef __cplusplus
}
#endif

#endif
