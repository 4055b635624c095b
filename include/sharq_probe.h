/*
 * sharq_probe.h -- a measurement aid, not part of the SharQ method.
 *
 * libsharq_probe.so runs back-to-back scaled FP4 MFMAs
 * (v_mfma_scale_f32_32x32x64_f8f6f4, E2M1 operands, unit E8M0 scales), or
 * bf16 or fp16 MFMAs, on every SIMD of the device and records the shader
 * clock.  The rate it reaches is the sustained matrix-core ceiling that bounds
 * a GEMM built on that instruction (the two-path MXFP4 GEMM on the FP4 one,
 * the NVFP4 GEMM on the fp16 one, the HiF4 GEMM and the NVFP4 GEMM for K not a
 * multiple of 64 on the bf16 one): under such load the part runs below
 * its rated clock, so this ceiling sits below the published dense peak.  The
 * benchmark reports each GEMM's rate against both.  Callers: the benchmark
 * and its tests.
 */
#ifndef SHARQ_PROBE_H
#define SHARQ_PROBE_H

#include <hip/hip_runtime.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Launch one workgroup of four wavefronts (one per SIMD) on each of
 * `workgroups` compute units (pass the device's CU count); every wavefront
 * issues iters x 32 independent FP4 MFMAs (8 accumulators, operand registers
 * cycled through four sets of pseudo-random E2M1 codes), then writes one float
 * per lane to `sink` (device, workgroups x 256 floats, contents meaningless)
 * and, from lane 0 of wavefront 0, two counters to `clk` (device,
 * workgroups x 2 uint64): shader-clock cycles and 100 MHz real-time ticks
 * between the first and the last MFMA.  Total work: workgroups x 4 x iters x 32
 * MFMAs of 2 x 32 x 32 x 64 flops.  Asynchronous on `stream`; time it with
 * events on that stream.
 * Returns hipSuccess, hipErrorInvalidValue (iters < 1, workgroups < 1, a NULL
 * pointer) or the launch error.
 */
int sharq_probe_mfma_fp4(int iters, int workgroups, float* sink, unsigned long long* clk, hipStream_t stream);

/*
 * The same for the bf16 MFMA (v_mfma_f32_32x32x16_bf16, pseudo-random finite
 * bf16 operands), the instruction the HiF4 GEMM and the NVFP4 GEMM for K not
 * a multiple of 64 run on: every wavefront issues iters x 32 independent
 * MFMAs of 2 x 32 x 32 x 16 flops.  Same arguments, outputs and errors as
 * sharq_probe_mfma_fp4.
 */
int sharq_probe_mfma_bf16(int iters, int workgroups, float* sink, unsigned long long* clk, hipStream_t stream);

/*
 * The same for the fp16 MFMA (v_mfma_f32_32x32x16_f16, pseudo-random finite
 * fp16 operands), the instruction of the NVFP4 GEMM for K a multiple of 64.
 * Same arguments, outputs and errors as sharq_probe_mfma_fp4.
 */
int sharq_probe_mfma_f16(int iters, int workgroups, float* sink, unsigned long long* clk, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif
