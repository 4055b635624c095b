"""Python binding of libsharq.so (the HIP kernels behind include/sharq.h).

Argument marshalling only: buffers are torch tensors on the GPU (torch is used
for device memory and streams), every computation runs in the library's
kernels.  Importing this module raises if the library has not been built;
there is no fallback path.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libsharq.so")

OK, EINVAL, EUNSUPPORTED, EALIGN, EHIP = 0, 1, 2, 3, 4
MXFP4, NVFP4, HIF4 = 0, 1, 2
BF16, F16, F32 = 0, 1, 2

_FMT = {"mx": MXFP4, "mxfp4": MXFP4, "nv": NVFP4, "nvfp4": NVFP4, "hif4": HIF4}
#: path combinations (sharq_mode): the method, and the ablation modes
MODES = {"sharq": 0, "sparse": 1, "dense": 2, "dense_dense": 3, "sparse_sparse": 4}
_DT = {torch.bfloat16: BF16, torch.float16: F16, torch.float32: F32}
#: E8M0 scale rules of MXFP4 (sharq_scale_rule)
SCALE_RULES = {"floor": 0, "ceil": 1}


class SharqError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {lib.sharq_status_str(status).decode()} (status {status})")


class Pattern(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("m", ctypes.c_int32), ("pairs", ctypes.c_int32)]


class ActStruct(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("K", ctypes.c_int64), ("fmt", ctypes.c_int), ("nm", Pattern),
                ("sp_codes", ctypes.c_void_p), ("sp_meta", ctypes.c_void_p), ("sp_scale", ctypes.c_void_p),
                ("dn_codes", ctypes.c_void_p), ("dn_scale", ctypes.c_void_p), ("tensor_scale", ctypes.c_void_p),
                ("mode", ctypes.c_int), ("dn_meta", ctypes.c_void_p), ("sp_dense", ctypes.c_void_p),
                ("scale_rule", ctypes.c_int), ("dbg_mask", ctypes.c_void_p), ("dbg_r", ctypes.c_void_p)]


class WeightStruct(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("K", ctypes.c_int64), ("experts", ctypes.c_int64), ("fmt", ctypes.c_int),
                ("codes", ctypes.c_void_p), ("scale", ctypes.c_void_p), ("scale_dn", ctypes.c_void_p),
                ("tensor_scale", ctypes.c_void_p), ("scale_rule", ctypes.c_int)]


def _load():
    if not os.path.exists(_LIB_PATH):
        raise ImportError(f"{_LIB_PATH} is not built; run `python -m paper_2606_26587_amd.build`")
    L = ctypes.CDLL(_LIB_PATH)
    c_i64, c_vp, c_f = ctypes.c_int64, ctypes.c_void_p, ctypes.c_float
    L.sharq_version.restype = ctypes.c_char_p
    L.sharq_version.argtypes = []
    L.sharq_status_str.restype = ctypes.c_char_p
    L.sharq_status_str.argtypes = [ctypes.c_int]
    L.sharq_act_buffer_bytes.restype = ctypes.c_size_t
    L.sharq_act_buffer_bytes.argtypes = [c_i64, c_i64, ctypes.c_int, Pattern, ctypes.c_int32]
    L.sharq_act_buffer_bytes_mode.restype = ctypes.c_size_t
    L.sharq_act_buffer_bytes_mode.argtypes = [c_i64, c_i64, ctypes.c_int, Pattern, ctypes.c_int, ctypes.c_int32]
    L.sharq_weight_buffer_bytes.restype = ctypes.c_size_t
    L.sharq_weight_buffer_bytes.argtypes = [c_i64, c_i64, ctypes.c_int, ctypes.c_int32]
    L.sharq_quantize_weight.restype = ctypes.c_int
    L.sharq_quantize_weight.argtypes = [c_vp, ctypes.c_int, c_i64, c_i64, c_i64, ctypes.POINTER(WeightStruct), c_vp]
    L.sharq_prepare.restype = ctypes.c_int
    L.sharq_prepare.argtypes = [c_vp, ctypes.c_int, c_i64, c_i64, c_i64, c_vp, c_f, Pattern, ctypes.c_int, c_vp,
                                ctypes.POINTER(ActStruct), c_vp]
    L.sharq_prepare_residual.restype = ctypes.c_int
    L.sharq_prepare_residual.argtypes = [c_vp, c_vp, c_vp, ctypes.c_int, c_i64, c_i64, c_i64, c_i64, c_i64, c_vp, c_f,
                                         Pattern, ctypes.c_int, c_vp, ctypes.POINTER(ActStruct), c_vp]
    L.sharq_prepare_silu_mul.restype = ctypes.c_int
    L.sharq_prepare_silu_mul.argtypes = [c_vp, c_vp, c_vp, ctypes.c_int, c_i64, c_i64, c_i64, c_i64, c_i64, Pattern,
                                         ctypes.c_int, c_vp, ctypes.POINTER(ActStruct), c_vp]
    L.sharq_linear.restype = ctypes.c_int
    L.sharq_linear.argtypes = [ctypes.POINTER(ActStruct), ctypes.POINTER(WeightStruct), c_vp, ctypes.c_int, c_i64,
                               c_vp]
    L.sharq_prepare_linear.restype = ctypes.c_int
    L.sharq_prepare_linear.argtypes = [c_vp, ctypes.c_int, c_i64, c_i64, c_i64, c_vp, c_f, Pattern, ctypes.c_int, c_vp,
                                       ctypes.POINTER(ActStruct), ctypes.POINTER(WeightStruct), c_vp, ctypes.c_int,
                                       c_i64, c_vp]
    L.sharq_linear_grouped.restype = ctypes.c_int
    L.sharq_linear_grouped.argtypes = [ctypes.POINTER(ActStruct), c_vp, c_vp, c_i64, ctypes.POINTER(WeightStruct),
                                       c_vp, ctypes.c_int, c_i64, c_vp]
    return L


lib = _load()


def _check(status: int, where: str):
    if status != OK:
        raise SharqError(status, where)


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream) -> ctypes.c_void_p:
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


# ---------------------------------------------------------------------------
# Containers
# ---------------------------------------------------------------------------

@dataclass
class PreparedAct:
    """Output of sharq_prepare: the compressed backbone and the residual (device
    buffers).  In the ablation modes path 1 lives in the sp_* buffers and path 2
    in the dn_* buffers (dn_meta: a sparse path 2)."""
    rows: int
    K: int
    fmt: int
    n: int
    m: int
    sp_codes: torch.Tensor
    sp_meta: torch.Tensor
    sp_scale: torch.Tensor
    dn_codes: torch.Tensor
    dn_scale: torch.Tensor
    tensor_scale: Optional[torch.Tensor] = None
    pairs: bool = False
    mode: int = 0
    dn_meta: Optional[torch.Tensor] = None
    sp_dense: Optional[torch.Tensor] = None   # MXFP4/NVFP4: the backbone's dense copy for the main GEMM
    scale_rule: int = 0                       # MXFP4: E8M0 rule (SCALE_RULES)
    dbg_mask: Optional[torch.Tensor] = None   # debug: keep bits, 4 bytes per 32 positions
    dbg_r: Optional[torch.Tensor] = None      # debug: RMSNorm r per row (fp32)

    def struct(self) -> ActStruct:
        def p(t):
            return None if t is None else t.data_ptr()
        return ActStruct(self.rows, self.K, self.fmt, Pattern(self.n, self.m, int(self.pairs)), p(self.sp_codes),
                         p(self.sp_meta), p(self.sp_scale), p(self.dn_codes), p(self.dn_scale), p(self.tensor_scale),
                         self.mode, p(self.dn_meta), p(self.sp_dense), self.scale_rule, p(self.dbg_mask),
                         p(self.dbg_r))


@dataclass
class QuantWeight:
    """Shared FP4 weight payload with its path-specific scale views (device buffers)."""
    N: int
    K: int
    experts: int
    fmt: int
    codes: torch.Tensor
    scale: torch.Tensor
    scale_dn: torch.Tensor
    tensor_scale: Optional[torch.Tensor] = None
    scale_rule: int = 0                       # MXFP4: E8M0 rule used by sharq_quantize_weight

    def struct(self) -> WeightStruct:
        return WeightStruct(self.N, self.K, self.experts, self.fmt, self.codes.data_ptr(), self.scale.data_ptr(),
                            self.scale_dn.data_ptr(),
                            None if self.tensor_scale is None else self.tensor_scale.data_ptr(), self.scale_rule)


def alloc_act(rows: int, K: int, n: int = 2, m: int = 4, fmt="mx", device="cuda", pairs: bool = False,
              mode="sharq", dense_backbone: bool = False, dense_only: bool = False, scale_rule="floor",
              debug: bool = False) -> PreparedAct:
    """Device buffers of a prepared activation (flat, panel-major; see include/sharq.h).
    pairs=True: n:m selection in pairs (4:8 in pairs).  mode: a key of MODES
    (or its id); buffers a mode does not use are empty.  dense_backbone=True
    (MXFP4, NVFP4): also the backbone's dense copy that the main GEMM reads without
    expanding it; dense_only=True: that copy instead of the compressed
    backbone.  scale_rule: "floor" or "ceil" (MXFP4 E8M0 rule).  debug=True:
    also the keep-mask and per-row r debug outputs."""
    f = _FMT[fmt] if isinstance(fmt, str) else fmt
    md = MODES[mode] if isinstance(mode, str) else int(mode)
    sizes = [lib.sharq_act_buffer_bytes_mode(rows, K, f, Pattern(n, m, int(pairs)), md, w) for w in range(6)]
    used = sizes[:5] if md == 0 else [z for z in sizes if z]
    if K <= 0 or K % 32 or (rows > 0 and (not used or min(used) == 0)):
        raise SharqError(EINVAL, "alloc_act")
    bufs = [torch.empty(sz, dtype=torch.uint8, device=device) for sz in sizes]
    ts = torch.empty(1, dtype=torch.float32, device=device) if f == NVFP4 else None
    spd = torch.empty(rows * K // 2, dtype=torch.uint8, device=device) if (dense_backbone or dense_only) else None
    if dense_only:
        bufs[0] = bufs[1] = None
    rule = SCALE_RULES[scale_rule] if isinstance(scale_rule, str) else int(scale_rule)
    dbg_mask = torch.empty(rows * K // 8, dtype=torch.uint8, device=device) if debug else None
    dbg_r = torch.empty(rows, dtype=torch.float32, device=device) if debug else None
    return PreparedAct(rows, K, f, n, m, *bufs[:5], tensor_scale=ts, pairs=pairs, mode=md, dn_meta=bufs[5],
                       sp_dense=spd, scale_rule=rule, dbg_mask=dbg_mask, dbg_r=dbg_r)


def alloc_weight(N: int, K: int, fmt="mx", experts: int = 1, device="cuda", scale_rule="floor") -> QuantWeight:
    """Device buffers of a quantized weight, one flat panel-major row per expert."""
    f = _FMT[fmt] if isinstance(fmt, str) else fmt
    codes = torch.empty((experts, N * K // 2), dtype=torch.uint8, device=device)
    scale = torch.empty((experts, N * K // (16 if f == HIF4 else 32)), dtype=torch.uint8, device=device)
    scale_dn = scale if f != NVFP4 else torch.empty((experts, N * K // 16), dtype=torch.uint8, device=device)
    ts = torch.empty(experts, dtype=torch.float32, device=device) if f == NVFP4 else None
    rule = SCALE_RULES[scale_rule] if isinstance(scale_rule, str) else int(scale_rule)
    return QuantWeight(N, K, experts, f, codes, scale, scale_dn, ts, rule)


# ---------------------------------------------------------------------------
# Entry points (same names as the C ABI)
# ---------------------------------------------------------------------------

def sharq_quantize_weight(w: torch.Tensor, fmt="mx", out: Optional[QuantWeight] = None, stream=None,
                          scale_rule="floor") -> QuantWeight:
    """Quantize W [N, K] (bf16 or fp32, on the GPU) into the shared FP4 payload
    (scale_rule: the MXFP4 E8M0 rule, ignored when `out` is given)."""
    N, K = w.shape
    if out is None:
        out = alloc_weight(N, K, fmt, 1, w.device, scale_rule)
    ws = out.struct()
    _check(lib.sharq_quantize_weight(_ptr(w), _DT.get(w.dtype, -1), N, K, w.stride(0), ctypes.byref(ws),
                                     _stream(stream)), "sharq_quantize_weight")
    return out


def sharq_prepare(x: torch.Tensor, gamma: Optional[torch.Tensor], eps: float = 1e-6, n: int = 2, m: int = 4,
                  fmt="mx", tensor_scale_in: Optional[torch.Tensor] = None, out: Optional[PreparedAct] = None,
                  stream=None, pairs: bool = False, mode="sharq", scale_rule="floor") -> PreparedAct:
    """Fused preparation of activation rows X [M, K] (bf16, on the GPU).
    pairs=True: n:m selection in pairs (NVFP4's 4:8 in pairs).  mode, scale_rule:
    the path combination (MODES) and the MXFP4 E8M0 rule (SCALE_RULES), both
    ignored when `out` is given, which carries them."""
    M, K = x.shape
    if out is None:
        out = alloc_act(M, K, n, m, fmt, x.device, pairs, mode, scale_rule=scale_rule)
    f = _FMT[fmt] if isinstance(fmt, str) else fmt
    st = out.struct()
    _check(lib.sharq_prepare(_ptr(x), _DT.get(x.dtype, -1), M, K, x.stride(0), _ptr(gamma), ctypes.c_float(eps),
                             Pattern(n, m, int(pairs)), f, _ptr(tensor_scale_in), ctypes.byref(st), _stream(stream)),
           "sharq_prepare")
    return out


def sharq_prepare_residual(x: torch.Tensor, residual: torch.Tensor, gamma: Optional[torch.Tensor], eps: float = 1e-6,
                           n: int = 2, m: int = 4, fmt="mx", h_out: Optional[torch.Tensor] = None,
                           tensor_scale_in: Optional[torch.Tensor] = None, out: Optional[PreparedAct] = None,
                           stream=None, pairs: bool = False):
    """Residual add fused into the preparation: h = bf16(x + residual) is
    written to h_out (a new tensor, or e.g. `residual` itself for an in-place
    update) and prepared.  Returns (prepared activation, h)."""
    M, K = x.shape
    if out is None:
        out = alloc_act(M, K, n, m, fmt, x.device, pairs)
    if h_out is None:
        h_out = torch.empty_like(x)
    f = _FMT[fmt] if isinstance(fmt, str) else fmt
    st = out.struct()
    _check(lib.sharq_prepare_residual(_ptr(x), _ptr(residual), _ptr(h_out), _DT.get(x.dtype, -1), M, K, x.stride(0),
                                      residual.stride(0), h_out.stride(0), _ptr(gamma), ctypes.c_float(eps),
                                      Pattern(n, m, int(pairs)), f, _ptr(tensor_scale_in), ctypes.byref(st),
                                      _stream(stream)), "sharq_prepare_residual")
    return out, h_out


def sharq_prepare_silu_mul(gate: torch.Tensor, up: torch.Tensor, n: int = 2, m: int = 4, fmt="mx",
                           h_out: Optional[torch.Tensor] = None, tensor_scale_in: Optional[torch.Tensor] = None,
                           out: Optional[PreparedAct] = None, stream=None, pairs: bool = False) -> PreparedAct:
    """SiLU.mul fused into the preparation of a down projection's input:
    h = bf16(SiLU(gate) * up) is prepared (and written to h_out when given)."""
    M, K = gate.shape
    if out is None:
        out = alloc_act(M, K, n, m, fmt, gate.device, pairs)
    f = _FMT[fmt] if isinstance(fmt, str) else fmt
    st = out.struct()
    _check(lib.sharq_prepare_silu_mul(_ptr(gate), _ptr(up), _ptr(h_out), _DT.get(gate.dtype, -1), M, K,
                                      gate.stride(0), up.stride(0), h_out.stride(0) if h_out is not None else K,
                                      Pattern(n, m, int(pairs)), f, _ptr(tensor_scale_in), ctypes.byref(st),
                                      _stream(stream)), "sharq_prepare_silu_mul")
    return out


def sharq_linear(a: PreparedAct, w: QuantWeight, out: Optional[torch.Tensor] = None, dtype=torch.bfloat16,
                 stream=None) -> torch.Tensor:
    """Y [rows, N] = backbone GEMM + residual GEMM over the shared weight."""
    if out is None:
        out = torch.empty((a.rows, w.N), dtype=dtype, device=a.dn_codes.device)
    ast, wst = a.struct(), w.struct()
    _check(lib.sharq_linear(ctypes.byref(ast), ctypes.byref(wst), _ptr(out), _DT.get(out.dtype, -1),
                            out.stride(0) if out.dim() == 2 else w.N, _stream(stream)), "sharq_linear")
    return out


def sharq_prepare_linear(x: torch.Tensor, gamma: Optional[torch.Tensor], w: QuantWeight, eps: float = 1e-6, n: int = 2,
                         m: int = 4, fmt="mx", act: Optional[PreparedAct] = None, out: Optional[torch.Tensor] = None,
                         dtype=torch.bfloat16, tensor_scale_in: Optional[torch.Tensor] = None, stream=None,
                         pairs: bool = False, scale_rule="floor"):
    """Preparation of X [M, K] into `act` and Y = SharQ(act, w) in one call
    (one kernel for a few rows).  Returns (prepared activation, Y)."""
    M, K = x.shape
    if act is None:
        act = alloc_act(M, K, n, m, fmt, x.device, pairs, scale_rule=scale_rule)
    if out is None:
        out = torch.empty((M, w.N), dtype=dtype, device=x.device)
    f = _FMT[fmt] if isinstance(fmt, str) else fmt
    ast, wst = act.struct(), w.struct()
    _check(lib.sharq_prepare_linear(_ptr(x), _DT.get(x.dtype, -1), M, K, x.stride(0), _ptr(gamma), ctypes.c_float(eps),
                                    Pattern(n, m, int(pairs)), f, _ptr(tensor_scale_in), ctypes.byref(ast),
                                    ctypes.byref(wst), _ptr(out), _DT.get(out.dtype, -1),
                                    out.stride(0) if out.dim() == 2 else w.N, _stream(stream)), "sharq_prepare_linear")
    return act, out


def sharq_linear_grouped(a: PreparedAct, row_index: Optional[torch.Tensor], expert_offsets: torch.Tensor, total: int,
                         w: QuantWeight, out: Optional[torch.Tensor] = None, dtype=torch.bfloat16,
                         stream=None) -> torch.Tensor:
    """Mixture-of-experts form: Y[i] = SharQ(A[row_index[i]], W_e) for i in expert e's slice."""
    if out is None:
        out = torch.empty((total, w.N), dtype=dtype, device=a.dn_codes.device)
    ast, wst = a.struct(), w.struct()
    _check(lib.sharq_linear_grouped(ctypes.byref(ast), _ptr(row_index), _ptr(expert_offsets), total,
                                    ctypes.byref(wst), _ptr(out), _DT.get(out.dtype, -1),
                                    out.stride(0) if out.dim() == 2 else w.N, _stream(stream)),
           "sharq_linear_grouped")
    return out


def stack_weights(ws: Sequence[QuantWeight]) -> QuantWeight:
    """Stack per-expert weights of one shape into one [experts] payload (device copies)."""
    w0 = ws[0]
    ts = None if w0.tensor_scale is None else torch.cat([w.tensor_scale for w in ws])
    scale = torch.cat([w.scale for w in ws])
    scale_dn = scale if w0.fmt != NVFP4 else torch.cat([w.scale_dn for w in ws])
    return QuantWeight(w0.N, w0.K, len(ws), w0.fmt, torch.cat([w.codes for w in ws]), scale, scale_dn, ts,
                       w0.scale_rule)


def version() -> str:
    return lib.sharq_version().decode()
