/*
 * sharq_ref.h -- plain C oracle of the SharQ sparse-dense MXFP4 linear layer
 * (SharQ, arXiv 2606.26587), TEST INFRASTRUCTURE ONLY.
 *
 * The host-pointer twin of the library's preparation, weight quantization and
 * two-path GEMM for MXFP4 (2:4 and 4:8 element-wise selection, optional
 * RMSNorm, floor or ceil E8M0 rule), written as straight scalar loops from the
 * paper's definitions and the readings the NumPy oracle lists (R1-R6, R13).
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

/* OpenMP threads used over rows (0 or negative: the runtime's default). */
void sharq_ref_set_threads(int threads);
int sharq_ref_max_threads(void);

#ifdef __cplusplus
}
#endif

#endif
