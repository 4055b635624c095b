// C ABI of the SharQ library: argument validation and kernel dispatch.  The
// entry points and their contracts are declared in include/sharq.h.

#include <limits.h>

#include "../../include/sharq.h"
#include "sharq_device.hpp"

namespace sharq {
hipError_t launch_prep(const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* res, int64_t ldr, uint16_t* h,
                       int64_t ldh, const uint16_t* gamma, float eps, int pat, bool nv, const float* ts_in,
                       float* ts_out, uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns,
                       uint8_t* spd, PrepExtras ex, hipStream_t st);
hipError_t launch_wquant_mx(const void* W, int wdt, int N, int K, int64_t ldw, uint8_t* codes, uint8_t* scale,
                            uint32_t rule_bias, hipStream_t st);
hipError_t launch_wquant_nv(const void* W, int wdt, int N, int K, int64_t ldw, uint8_t* codes, uint8_t* scale,
                            uint8_t* scale_dn, float* ts, hipStream_t st);
hipError_t launch_linear_nv(int pat, int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps,
                            const uint8_t* dnc, const uint8_t* dns, const float* tsx, int64_t M, const uint8_t* wc,
                            const uint8_t* ws, const float* tsw, int N, int K, void* Y, int64_t ldy,
                            const uint8_t* spd, hipStream_t st);
hipError_t launch_linear_mx(int pat, int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps,
                            const uint8_t* dnc, const uint8_t* dns, int64_t M, const uint8_t* wc, const uint8_t* ws,
                            int N, int K, void* Y, int64_t ldy, const uint8_t* spd, hipStream_t st);
hipError_t launch_prep_mode(int mode, const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* gamma, float eps,
                            int pat, bool nv, const float* ts_in, float* ts_out, uint8_t* c1, uint8_t* m1,
                            uint8_t* s1, uint8_t* c2, uint8_t* m2, uint8_t* s2, hipStream_t st);
hipError_t launch_linear_slots(int mode, int pat, int ydt, bool nv, const uint8_t* c1, const uint8_t* m1,
                               const uint8_t* s1, const uint8_t* c2, const uint8_t* m2, const uint8_t* s2,
                               const float* tsx, int64_t M, const uint8_t* wc, const uint8_t* ws, const float* tsw,
                               int N, int K, void* Y, int64_t ldy, hipStream_t st);
hipError_t launch_prep_hif4(const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* gamma, float eps,
                            uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns, hipStream_t st);
hipError_t launch_wquant_hif4(const void* W, int wdt, int N, int K, int64_t ldw, uint8_t* codes, uint8_t* scale,
                              hipStream_t st);
hipError_t launch_linear_hif4(int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps, const uint8_t* dnc,
                              const uint8_t* dns, int64_t M, const uint8_t* wc, const uint8_t* ws, int N, int K,
                              void* Y, int64_t ldy, hipStream_t st);
hipError_t launch_prep_silu(const uint16_t* gate, const uint16_t* up, uint16_t* h, int M, int K, int64_t ldg,
                            int64_t ldu, int64_t ldh, int pat, bool nv, const float* ts_in, float* ts_out,
                            uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns, uint8_t* spd,
                            PrepExtras ex, hipStream_t st);
bool fused_prep_linear_applies(int64_t M, int K, int N);
hipError_t launch_prep_linear_fused(const uint16_t* X, int M, int K, int64_t ldx, const uint16_t* gamma, float eps,
                                    int pat, uint8_t* spc, uint8_t* spm, uint8_t* sps, uint8_t* dnc, uint8_t* dns,
                                    uint8_t* spd, PrepExtras ex, const uint8_t* wc, const uint8_t* ws, int N, int ydt,
                                    void* Y, int64_t ldy, hipStream_t st);
hipError_t launch_linear_mx_grouped(int pat, int ydt, const uint8_t* spc, const uint8_t* spm, const uint8_t* sps,
                                    const uint8_t* dnc, const uint8_t* dns, const int32_t* ridx, int64_t act_rows,
                                    const int32_t* offs, int E, int64_t total, const uint8_t* wc, const uint8_t* ws,
                                    int N, int K, void* Y, int64_t ldy, const uint8_t* spd, hipStream_t st);
}  // namespace sharq

namespace {

constexpr int64_t kMaxK = 1 << 20;
constexpr int64_t kMaxNormK = 16384;   // RMSNorm rows are held in registers
constexpr int kMaxExperts = 1024;

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// 24 for 2:4, 48 for 4:8, 49 for 4:8 in pairs, 0 if the pattern is valid but
// not built, -1 if invalid
int pattern_id(sharq_pattern nm) {
  if (nm.m <= 0 || nm.n < 0 || nm.n > nm.m || (nm.pairs != 0 && nm.pairs != 1)) return -1;
  if (nm.pairs && (nm.m % 2 != 0 || nm.n % 2 != 0)) return -1;
  if (!nm.pairs && nm.n == 2 && nm.m == 4) return 24;
  if (nm.n == 4 && nm.m == 8) return nm.pairs ? 49 : 48;
  return 0;
}

// The GEMMs read the metadata only: 4:8 in pairs has the 4:8 keep-mask layout.
int gemm_pattern(int pid) { return pid == 49 ? 48 : pid; }

sharq_status hip_status(hipError_t e) { return e == hipSuccess ? SHARQ_OK : SHARQ_EHIP; }

bool fmt_ok(int f) { return f == SHARQ_MXFP4 || f == SHARQ_NVFP4 || f == SHARQ_HIF4; }

// Path kinds of the two slots of a mode: 0 absent, 1 sparse, 2 dense.
constexpr int kNone = 0, kSparse = 1, kDense = 2;
bool mode_ok(int mode) { return mode >= SHARQ_MODE_SHARQ && mode <= SHARQ_MODE_SPARSE_SPARSE; }
int kind1(int mode) { return mode == SHARQ_MODE_DENSE ? kNone : (mode == SHARQ_MODE_DENSE_DENSE ? kDense : kSparse); }
int kind2(int mode) {
  return mode == SHARQ_MODE_SPARSE ? kNone : (mode == SHARQ_MODE_SPARSE_SPARSE ? kSparse : kDense);
}
bool has_sparse(int mode) { return kind1(mode) == kSparse || kind2(mode) == kSparse; }

// Row bytes per 32 K positions of a slot's codes / metadata / scales.
size_t slot_bytes(int kind, sharq_pattern nm, sharq_format fmt, int what, size_t k) {
  if (kind == kNone) return 0;
  if (kind == kSparse)
    return what == 0 ? k * (size_t)nm.n / (size_t)nm.m / 2 : what == 1 ? k / 8 : (fmt == SHARQ_HIF4 ? k / 16 : k / 32);
  return what == 0 ? k / 2 : what == 1 ? 0 : (fmt == SHARQ_MXFP4 ? k / 32 : k / 16);
}

sharq_status check_act(const sharq_act* a) {
  if (!a) return SHARQ_EINVAL;
  if (a->rows < 0 || a->rows > INT_MAX || a->K <= 0 || a->K % 32 != 0 || a->K > kMaxK) return SHARQ_EINVAL;
  if (!mode_ok((int)a->mode)) return SHARQ_EINVAL;
  const int mode = (int)a->mode;
  const int pid = pattern_id(a->nm);   // 0: valid, not built
  if (pid < 0 || a->K % a->nm.m != 0) return SHARQ_EINVAL;
  if (pid == 0 && has_sparse(mode)) return SHARQ_EUNSUPPORTED;
  if (!fmt_ok(a->fmt)) return SHARQ_EINVAL;
  if (a->fmt == SHARQ_HIF4) {   // built: 2:4 backbone, the method's path combination
    if (a->K % 64 != 0) return SHARQ_EINVAL;
    if (pid != 24 || mode != SHARQ_MODE_SHARQ) return SHARQ_EUNSUPPORTED;
  }
  if (a->scale_rule != SHARQ_SCALE_FLOOR && a->scale_rule != SHARQ_SCALE_CEIL) return SHARQ_EINVAL;
  if (a->scale_rule == SHARQ_SCALE_CEIL && (a->fmt != SHARQ_MXFP4 || mode != SHARQ_MODE_SHARQ))
    return SHARQ_EUNSUPPORTED;
  if ((a->dbg_mask || a->dbg_r) && (a->fmt == SHARQ_HIF4 || mode != SHARQ_MODE_SHARQ)) return SHARQ_EUNSUPPORTED;
  if (a->rows == 0) return SHARQ_OK;   // an empty activation is never dereferenced
  const int k1 = kind1(mode), k2 = kind2(mode);
  // the dense-only backbone: sp_dense without the compressed codes and metadata
  const bool dense_only = a->sp_dense && !a->sp_codes && !a->sp_meta && mode == SHARQ_MODE_SHARQ;
  if (dense_only && (a->fmt == SHARQ_HIF4 || a->K % 128 != 0)) return SHARQ_EUNSUPPORTED;
  if (k1 != kNone && !dense_only && (!a->sp_codes || !a->sp_scale || (k1 == kSparse && !a->sp_meta)))
    return SHARQ_EINVAL;
  if (dense_only && !a->sp_scale) return SHARQ_EINVAL;
  if (k2 != kNone && (!a->dn_codes || !a->dn_scale)) return SHARQ_EINVAL;
  if (k2 == kSparse && !a->dn_meta) return SHARQ_EINVAL;
  if (a->fmt == SHARQ_NVFP4 && !a->tensor_scale) return SHARQ_EINVAL;
  if (a->sp_dense && (a->fmt == SHARQ_HIF4 || mode != SHARQ_MODE_SHARQ)) return SHARQ_EUNSUPPORTED;
  if (!aligned(a->sp_dense, 16)) return SHARQ_EALIGN;
  if (!aligned(a->sp_codes, 16) || !aligned(a->dn_codes, 16) || !aligned(a->sp_meta, 4) ||
      !aligned(a->sp_scale, 4) || !aligned(a->dn_scale, 4) || !aligned(a->tensor_scale, 4) ||
      !aligned(a->dn_meta, 4) || !aligned(a->dbg_mask, 4) || !aligned(a->dbg_r, 4))
    return SHARQ_EALIGN;
  return SHARQ_OK;
}

uint32_t rule_bias(sharq_scale_rule r) { return r == SHARQ_SCALE_CEIL ? sharq::kE8Ceil : sharq::kE8Floor; }

sharq_status check_weight(const sharq_weight* w) {
  if (!w) return SHARQ_EINVAL;
  if (w->N < 0 || w->N > INT_MAX || w->K <= 0 || w->K % 32 != 0 || w->K > kMaxK || w->experts < 1 ||
      w->experts > kMaxExperts)
    return SHARQ_EINVAL;
  if (!fmt_ok(w->fmt)) return SHARQ_EINVAL;
  if (w->fmt == SHARQ_HIF4 && w->K % 64 != 0) return SHARQ_EINVAL;
  if (!w->codes || !w->scale) return SHARQ_EINVAL;
  if (w->fmt == SHARQ_NVFP4 && (!w->scale_dn || !w->tensor_scale)) return SHARQ_EINVAL;
  if (!aligned(w->codes, 16) || !aligned(w->scale, 4) || !aligned(w->tensor_scale, 4)) return SHARQ_EALIGN;
  return SHARQ_OK;
}

bool ydt_ok(sharq_dtype d) { return d == SHARQ_BF16 || d == SHARQ_F16 || d == SHARQ_F32; }
size_t ysize(sharq_dtype d) { return d == SHARQ_F32 ? 4 : 2; }

}  // namespace

extern "C" {

const char* sharq_version(void) { return "sharq-gfx950 0.1"; }

const char* sharq_status_str(sharq_status s) {
  switch (s) {
    case SHARQ_OK: return "ok";
    case SHARQ_EINVAL: return "invalid argument";
    case SHARQ_EUNSUPPORTED: return "unsupported format/pattern/dtype combination";
    case SHARQ_EALIGN: return "misaligned pointer or leading dimension";
    case SHARQ_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

size_t sharq_act_buffer_bytes(int64_t rows, int64_t K, sharq_format fmt, sharq_pattern nm, int32_t which) {
  if (which < 0 || which > 4) return 0;
  return sharq_act_buffer_bytes_mode(rows, K, fmt, nm, SHARQ_MODE_SHARQ, which);
}

size_t sharq_act_buffer_bytes_mode(int64_t rows, int64_t K, sharq_format fmt, sharq_pattern nm, sharq_mode mode,
                                   int32_t which) {
  if (rows < 0 || K <= 0 || K % 32 != 0 || !mode_ok((int)mode)) return 0;
  const int pid = pattern_id(nm);
  if (pid < 0 || K % nm.m != 0 || (pid == 0 && has_sparse((int)mode))) return 0;
  if (!fmt_ok(fmt) || (fmt == SHARQ_HIF4 && K % 64 != 0)) return 0;
  const size_t r = (size_t)rows, k = (size_t)K;
  const int k1 = kind1((int)mode), k2 = kind2((int)mode);
  switch (which) {
    case 0: return r * slot_bytes(k1, nm, fmt, 0, k);
    case 1: return r * slot_bytes(k1, nm, fmt, 1, k);
    case 2: return r * slot_bytes(k1, nm, fmt, 2, k);
    case 3: return r * slot_bytes(k2, nm, fmt, 0, k);
    case 4: return r * slot_bytes(k2, nm, fmt, 2, k);
    case 5: return r * slot_bytes(k2, nm, fmt, 1, k);
    default: return 0;
  }
}

size_t sharq_weight_buffer_bytes(int64_t N, int64_t K, sharq_format fmt, int32_t which) {
  if (N < 0 || K <= 0 || K % 32 != 0) return 0;
  if (!fmt_ok(fmt) || (fmt == SHARQ_HIF4 && K % 64 != 0)) return 0;
  const size_t n = (size_t)N, k = (size_t)K;
  switch (which) {
    case 0: return n * (k / 2);
    case 1: return n * (fmt == SHARQ_HIF4 ? k / 16 : k / 32);
    case 2: return n * (fmt == SHARQ_MXFP4 ? k / 32 : k / 16);
    default: return 0;
  }
}

sharq_status sharq_quantize_weight(const void* W, sharq_dtype wdt, int64_t N, int64_t K, int64_t ldw,
                                   sharq_weight* out, void* stream) {
  if (!W || !out) return SHARQ_EINVAL;
  if (N < 0 || N > INT_MAX || K <= 0 || K % 32 != 0 || K > kMaxK || ldw < K) return SHARQ_EINVAL;
  if (out->N != N || out->K != K || out->experts != 1) return SHARQ_EINVAL;
  if (wdt != SHARQ_BF16 && wdt != SHARQ_F32) return SHARQ_EUNSUPPORTED;
  if (!fmt_ok(out->fmt)) return SHARQ_EINVAL;
  if (out->fmt == SHARQ_HIF4 && K % 64 != 0) return SHARQ_EINVAL;
  if (out->scale_rule != SHARQ_SCALE_FLOOR && out->scale_rule != SHARQ_SCALE_CEIL) return SHARQ_EINVAL;
  if (out->scale_rule == SHARQ_SCALE_CEIL && out->fmt != SHARQ_MXFP4) return SHARQ_EUNSUPPORTED;
  const bool nv = out->fmt == SHARQ_NVFP4;
  if (!out->codes || !out->scale) return SHARQ_EINVAL;
  if (nv && (!out->scale_dn || !out->tensor_scale)) return SHARQ_EINVAL;
  if (!aligned(W, 16) || (ldw * (int64_t)(wdt == SHARQ_F32 ? 4 : 2)) % 16 != 0 || !aligned(out->codes, 16) ||
      !aligned(out->tensor_scale, 4))
    return SHARQ_EALIGN;
  if (N == 0) return SHARQ_OK;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (out->fmt == SHARQ_HIF4)
    return hip_status(sharq::launch_wquant_hif4(W, (int)wdt, (int)N, (int)K, ldw, out->codes, out->scale, st));
  if (nv)
    return hip_status(sharq::launch_wquant_nv(W, (int)wdt, (int)N, (int)K, ldw, out->codes, out->scale,
                                              out->scale_dn, out->tensor_scale, st));
  return hip_status(sharq::launch_wquant_mx(W, (int)wdt, (int)N, (int)K, ldw, out->codes, out->scale,
                                            rule_bias(out->scale_rule), st));
}

}  // extern "C"

namespace {

// Shared by sharq_prepare, sharq_prepare_residual and sharq_prepare_silu_mul.
// Source kinds: 0, X itself; 1, the residual add (res = the residual, h_out
// required); 2, SiLU.mul (X = gate, res = up, h_out optional, no gamma).
constexpr int kSrcPlain = 0, kSrcResidual = 1, kSrcSilu = 2;

// check_only: validate the arguments and return before any launch.
sharq_status prepare_impl(int src, const void* X, const void* res, void* h_out, sharq_dtype xdt, int64_t M,
                          int64_t K, int64_t ldx, int64_t ldr, int64_t ldh, const void* gamma, float eps,
                          sharq_pattern nm, sharq_format fmt, const float* tensor_scale_in, sharq_act* out,
                          void* stream, bool check_only = false) {
  if (!out) return SHARQ_EINVAL;
  if (M < 0 || M > INT_MAX || K <= 0 || K % 32 != 0 || K > kMaxK || ldx < K) return SHARQ_EINVAL;
  if (!X && M > 0) return SHARQ_EINVAL;
  if (src == kSrcResidual && (ldr < K || ldh < K || (!h_out && M > 0))) return SHARQ_EINVAL;
  if (src == kSrcSilu && (ldr < K || (h_out && ldh < K) || gamma)) return SHARQ_EINVAL;
  const int pid = pattern_id(nm);
  if (pid < 0 || K % nm.m != 0) return SHARQ_EINVAL;
  if (out->rows != M || out->K != K || out->fmt != fmt || out->nm.n != nm.n || out->nm.m != nm.m ||
      out->nm.pairs != nm.pairs)
    return SHARQ_EINVAL;
  if (xdt != SHARQ_BF16) return SHARQ_EUNSUPPORTED;
  if (!(eps >= 0.0f)) return SHARQ_EINVAL;
  sharq_status s = check_act(out);
  if (s != SHARQ_OK) return s;
  if (gamma && K > kMaxNormK) return SHARQ_EUNSUPPORTED;
  const bool nv = fmt == SHARQ_NVFP4;
  if (nv && M > 0 && !out->tensor_scale) return SHARQ_EINVAL;
  if (!aligned(X, 16) || (ldx * 2) % 16 != 0 || (gamma && !aligned(gamma, 16)) || !aligned(tensor_scale_in, 4))
    return SHARQ_EALIGN;
  if (res && (!aligned(res, 16) || !aligned(h_out, 16) || (ldr * 2) % 16 != 0 || (h_out && (ldh * 2) % 16 != 0)))
    return SHARQ_EALIGN;
  if (res && out->mode != SHARQ_MODE_SHARQ) return SHARQ_EUNSUPPORTED;
  if (res && fmt == SHARQ_HIF4) return SHARQ_EUNSUPPORTED;
  if (M == 0 || check_only) return SHARQ_OK;
  const sharq::PrepExtras ex{rule_bias(out->scale_rule), reinterpret_cast<uint32_t*>(out->dbg_mask), out->dbg_r};
  if (src == kSrcSilu)
    return hip_status(sharq::launch_prep_silu(static_cast<const uint16_t*>(X), static_cast<const uint16_t*>(res),
                                              static_cast<uint16_t*>(h_out), (int)M, (int)K, ldx, ldr, ldh, pid, nv,
                                              nv ? tensor_scale_in : nullptr, nv ? out->tensor_scale : nullptr,
                                              out->sp_codes, out->sp_meta, out->sp_scale, out->dn_codes,
                                              out->dn_scale, out->sp_dense, ex, reinterpret_cast<hipStream_t>(stream)));
  if (fmt == SHARQ_HIF4)
    return hip_status(sharq::launch_prep_hif4(static_cast<const uint16_t*>(X), (int)M, (int)K, ldx,
                                              static_cast<const uint16_t*>(gamma), eps, out->sp_codes, out->sp_meta,
                                              out->sp_scale, out->dn_codes, out->dn_scale,
                                              reinterpret_cast<hipStream_t>(stream)));
  const int mode = (int)out->mode;
  if (mode != SHARQ_MODE_SHARQ) {
    if (res) return SHARQ_EUNSUPPORTED;
    return hip_status(sharq::launch_prep_mode(mode, static_cast<const uint16_t*>(X), (int)M, (int)K, ldx,
                                              static_cast<const uint16_t*>(gamma), eps, pid, nv,
                                              nv ? tensor_scale_in : nullptr, nv ? out->tensor_scale : nullptr,
                                              out->sp_codes, out->sp_meta, out->sp_scale, out->dn_codes,
                                              out->dn_meta, out->dn_scale, reinterpret_cast<hipStream_t>(stream)));
  }
  return hip_status(sharq::launch_prep(static_cast<const uint16_t*>(X), (int)M, (int)K, ldx,
                                       static_cast<const uint16_t*>(res), ldr, static_cast<uint16_t*>(h_out), ldh,
                                       static_cast<const uint16_t*>(gamma), eps, pid, nv, nv ? tensor_scale_in : nullptr,
                                       nv ? out->tensor_scale : nullptr, out->sp_codes, out->sp_meta, out->sp_scale,
                                       out->dn_codes, out->dn_scale, out->sp_dense, ex,
                                       reinterpret_cast<hipStream_t>(stream)));
}

}  // namespace

extern "C" {

sharq_status sharq_prepare(const void* X, sharq_dtype xdt, int64_t M, int64_t K, int64_t ldx, const void* gamma,
                           float eps, sharq_pattern nm, sharq_format fmt, const float* tensor_scale_in,
                           sharq_act* out, void* stream) {
  return prepare_impl(kSrcPlain, X, nullptr, nullptr, xdt, M, K, ldx, K, K, gamma, eps, nm, fmt, tensor_scale_in, out,
                      stream);
}

sharq_status sharq_prepare_residual(const void* X, const void* residual, void* h_out, sharq_dtype xdt, int64_t M,
                                    int64_t K, int64_t ldx, int64_t ldr, int64_t ldh, const void* gamma, float eps,
                                    sharq_pattern nm, sharq_format fmt, const float* tensor_scale_in,
                                    sharq_act* out, void* stream) {
  if (!residual && M > 0) return SHARQ_EINVAL;
  if (M == 0) residual = nullptr;
  return prepare_impl(kSrcResidual, X, residual, h_out, xdt, M, K, ldx, ldr, ldh, gamma, eps, nm, fmt,
                      tensor_scale_in, out, stream);
}

sharq_status sharq_prepare_silu_mul(const void* gate, const void* up, void* h_out, sharq_dtype xdt, int64_t M,
                                    int64_t K, int64_t ldg, int64_t ldu, int64_t ldh, sharq_pattern nm,
                                    sharq_format fmt, const float* tensor_scale_in, sharq_act* out, void* stream) {
  if (!up && M > 0) return SHARQ_EINVAL;
  if (M == 0) up = nullptr;
  return prepare_impl(kSrcSilu, gate, up, h_out, xdt, M, K, ldg, ldu, ldh, nullptr, 0.0f, nm, fmt, tensor_scale_in,
                      out, stream);
}

}  // extern "C"

namespace {

sharq_status check_linear(const sharq_act* a, const sharq_weight* w, const void* Y, sharq_dtype ydt, int64_t ldy) {
  sharq_status s = check_act(a);
  if (s != SHARQ_OK) return s;
  if (!Y && a->rows > 0) return SHARQ_EINVAL;
  s = check_weight(w);
  if (s != SHARQ_OK) return s;
  if (a->fmt != w->fmt || a->K != w->K || w->experts != 1) return SHARQ_EINVAL;
  if (!ydt_ok(ydt)) return SHARQ_EUNSUPPORTED;
  if (ldy < w->N) return SHARQ_EINVAL;
  if (!aligned(Y, ysize(ydt))) return SHARQ_EALIGN;
  return SHARQ_OK;
}

}  // namespace

extern "C" {

sharq_status sharq_linear(const sharq_act* a, const sharq_weight* w, void* Y, sharq_dtype ydt, int64_t ldy,
                          void* stream) {
  const sharq_status s = check_linear(a, w, Y, ydt, ldy);
  if (s != SHARQ_OK) return s;
  if (a->rows == 0 || w->N == 0) return SHARQ_OK;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (a->fmt == SHARQ_HIF4)
    return hip_status(sharq::launch_linear_hif4((int)ydt, a->sp_codes, a->sp_meta, a->sp_scale, a->dn_codes,
                                                a->dn_scale, a->rows, w->codes, w->scale, (int)w->N, (int)w->K, Y,
                                                ldy, st));
  if (a->mode != SHARQ_MODE_SHARQ) {
    const int pid = pattern_id(a->nm);
    return hip_status(sharq::launch_linear_slots((int)a->mode, pid > 0 ? gemm_pattern(pid) : 24, (int)ydt,
                                                 a->fmt == SHARQ_NVFP4, a->sp_codes, a->sp_meta, a->sp_scale,
                                                 a->dn_codes, a->dn_meta, a->dn_scale, a->tensor_scale, a->rows,
                                                 w->codes, w->scale, w->tensor_scale, (int)w->N, (int)w->K, Y, ldy,
                                                 st));
  }
  if (a->fmt == SHARQ_NVFP4)
    return hip_status(sharq::launch_linear_nv(gemm_pattern(pattern_id(a->nm)), (int)ydt, a->sp_codes, a->sp_meta, a->sp_scale,
                                              a->dn_codes, a->dn_scale, a->tensor_scale, a->rows, w->codes,
                                              w->scale, w->tensor_scale, (int)w->N, (int)w->K, Y, ldy,
                                              a->sp_dense, st));
  return hip_status(sharq::launch_linear_mx(gemm_pattern(pattern_id(a->nm)), (int)ydt, a->sp_codes, a->sp_meta, a->sp_scale,
                                            a->dn_codes, a->dn_scale, a->rows, w->codes, w->scale, (int)w->N,
                                            (int)w->K, Y, ldy, a->sp_dense, st));
}

sharq_status sharq_prepare_linear(const void* X, sharq_dtype xdt, int64_t M, int64_t K, int64_t ldx, const void* gamma,
                                  float eps, sharq_pattern nm, sharq_format fmt, const float* tensor_scale_in,
                                  sharq_act* act, const sharq_weight* w, void* Y, sharq_dtype ydt, int64_t ldy,
                                  void* stream) {
  // every argument of both steps is validated before anything is launched
  sharq_status s = prepare_impl(kSrcPlain, X, nullptr, nullptr, xdt, M, K, ldx, K, K, gamma, eps, nm, fmt,
                                tensor_scale_in, act, stream, true);
  if (s != SHARQ_OK) return s;
  s = check_linear(act, w, Y, ydt, ldy);
  if (s != SHARQ_OK) return s;
  if (M == 0 || w->N == 0) {
    if (M == 0) return SHARQ_OK;
    return prepare_impl(kSrcPlain, X, nullptr, nullptr, xdt, M, K, ldx, K, K, gamma, eps, nm, fmt, tensor_scale_in,
                        act, stream);
  }
  const int pid = pattern_id(nm);
  if (fmt == SHARQ_MXFP4 && act->mode == SHARQ_MODE_SHARQ && pid > 0 &&
      sharq::fused_prep_linear_applies(M, (int)K, (int)w->N)) {
    const sharq::PrepExtras ex{rule_bias(act->scale_rule), reinterpret_cast<uint32_t*>(act->dbg_mask), act->dbg_r};
    return hip_status(sharq::launch_prep_linear_fused(
        static_cast<const uint16_t*>(X), (int)M, (int)K, ldx, static_cast<const uint16_t*>(gamma), eps, pid,
        act->sp_codes, act->sp_meta, act->sp_scale, act->dn_codes, act->dn_scale, act->sp_dense, ex, w->codes,
        w->scale, (int)w->N, (int)ydt, Y, ldy, reinterpret_cast<hipStream_t>(stream)));
  }
  s = prepare_impl(kSrcPlain, X, nullptr, nullptr, xdt, M, K, ldx, K, K, gamma, eps, nm, fmt, tensor_scale_in, act,
                   stream);
  if (s != SHARQ_OK) return s;
  return sharq_linear(act, w, Y, ydt, ldy, stream);
}

sharq_status sharq_linear_grouped(const sharq_act* a, const int32_t* row_index, const int32_t* expert_offsets,
                                  int64_t total, const sharq_weight* w, void* Y, sharq_dtype ydt, int64_t ldy,
                                  void* stream) {
  if (!expert_offsets) return SHARQ_EINVAL;
  sharq_status s = check_act(a);
  if (s != SHARQ_OK) return s;
  if (!Y && total > 0) return SHARQ_EINVAL;
  s = check_weight(w);
  if (s != SHARQ_OK) return s;
  if (a->fmt != w->fmt || a->K != w->K) return SHARQ_EINVAL;
  if (a->fmt != SHARQ_MXFP4 || a->mode != SHARQ_MODE_SHARQ) return SHARQ_EUNSUPPORTED;
  if (total < 0 || total > INT_MAX) return SHARQ_EINVAL;
  if (!row_index && total > a->rows) return SHARQ_EINVAL;
  if (!ydt_ok(ydt)) return SHARQ_EUNSUPPORTED;
  if (ldy < w->N) return SHARQ_EINVAL;
  if (!aligned(Y, ysize(ydt)) || !aligned(expert_offsets, 4) || (row_index && !aligned(row_index, 4)))
    return SHARQ_EALIGN;
  if (total == 0 || w->N == 0) return SHARQ_OK;
  return hip_status(sharq::launch_linear_mx_grouped(
      gemm_pattern(pattern_id(a->nm)), (int)ydt, a->sp_codes, a->sp_meta, a->sp_scale, a->dn_codes, a->dn_scale, row_index,
      a->rows, expert_offsets, (int)w->experts, total, w->codes, w->scale, (int)w->N, (int)w->K, Y, ldy,
      a->sp_dense, reinterpret_cast<hipStream_t>(stream)));
}

}  // extern "C"
