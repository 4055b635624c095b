"""The C-ABI library loads, exports every declared entry point, sizes buffers
and rejects bad arguments -- all without a GPU (no call here launches work)."""

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2606_26587_amd", "libsharq.so")
HEADER = os.path.join(ROOT, "include", "sharq.h")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libsharq.so not built")

OK, EINVAL, EUNSUPPORTED, EALIGN = 0, 1, 2, 3


class Pattern(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int32), ("m", ctypes.c_int32), ("pairs", ctypes.c_int32)]


class Act(ctypes.Structure):
    _fields_ = [("rows", ctypes.c_int64), ("K", ctypes.c_int64), ("fmt", ctypes.c_int), ("nm", Pattern),
                ("sp_codes", ctypes.c_void_p), ("sp_meta", ctypes.c_void_p), ("sp_scale", ctypes.c_void_p),
                ("dn_codes", ctypes.c_void_p), ("dn_scale", ctypes.c_void_p), ("tensor_scale", ctypes.c_void_p),
                ("mode", ctypes.c_int), ("dn_meta", ctypes.c_void_p), ("sp_dense", ctypes.c_void_p),
                ("scale_rule", ctypes.c_int), ("dbg_mask", ctypes.c_void_p), ("dbg_r", ctypes.c_void_p)]


class Weight(ctypes.Structure):
    _fields_ = [("N", ctypes.c_int64), ("K", ctypes.c_int64), ("experts", ctypes.c_int64), ("fmt", ctypes.c_int),
                ("codes", ctypes.c_void_p), ("scale", ctypes.c_void_p), ("scale_dn", ctypes.c_void_p),
                ("tensor_scale", ctypes.c_void_p), ("scale_rule", ctypes.c_int)]


@pytest.fixture(scope="module")
def L():
    lib = ctypes.CDLL(LIB)
    lib.sharq_prepare.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                  ctypes.c_void_p, ctypes.c_float, Pattern, ctypes.c_int, ctypes.c_void_p,
                                  ctypes.POINTER(Act), ctypes.c_void_p]
    lib.sharq_prepare_residual.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                           ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                           ctypes.c_int64, ctypes.c_void_p, ctypes.c_float, Pattern, ctypes.c_int,
                                           ctypes.c_void_p, ctypes.POINTER(Act), ctypes.c_void_p]
    lib.sharq_linear.argtypes = [ctypes.POINTER(Act), ctypes.POINTER(Weight), ctypes.c_void_p, ctypes.c_int,
                                 ctypes.c_int64, ctypes.c_void_p]
    lib.sharq_linear_grouped.argtypes = [ctypes.POINTER(Act), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.POINTER(Weight), ctypes.c_void_p, ctypes.c_int, ctypes.c_int64,
                                         ctypes.c_void_p]
    lib.sharq_quantize_weight.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int64, ctypes.POINTER(Weight), ctypes.c_void_p]
    lib.sharq_act_buffer_bytes.restype = ctypes.c_size_t
    lib.sharq_act_buffer_bytes.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int, Pattern, ctypes.c_int32]
    lib.sharq_act_buffer_bytes_mode.restype = ctypes.c_size_t
    lib.sharq_act_buffer_bytes_mode.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int, Pattern, ctypes.c_int,
                                                ctypes.c_int32]
    lib.sharq_weight_buffer_bytes.restype = ctypes.c_size_t
    lib.sharq_weight_buffer_bytes.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_int32]
    lib.sharq_status_str.restype = ctypes.c_char_p
    lib.sharq_version.restype = ctypes.c_char_p
    return lib


def declared_functions():
    txt = open(HEADER).read()
    return re.findall(r"SHARQ_API\s+[\w\s\*]+?\b(sharq_\w+)\s*\(", txt)


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert {"sharq_quantize_weight", "sharq_prepare", "sharq_linear", "sharq_linear_grouped"} <= set(names)
    for n in names:
        assert hasattr(L, n), n
    assert L.sharq_version().startswith(b"sharq")
    assert L.sharq_status_str(2) == b"unsupported format/pattern/dtype combination"


def test_buffer_sizes(L):
    rows, K = 7, 4096
    mx = [L.sharq_act_buffer_bytes(rows, K, 0, Pattern(2, 4), w) for w in range(5)]
    assert mx == [rows * K // 4, rows * K // 8, rows * K // 32, rows * K // 2, rows * K // 32]
    nv = [L.sharq_act_buffer_bytes(rows, K, 1, Pattern(4, 8), w) for w in range(5)]
    assert nv[4] == rows * K // 16 and nv[0] == rows * K // 4
    assert L.sharq_act_buffer_bytes(rows, 100, 0, Pattern(2, 4), 0) == 0
    # 4:8 in pairs has the 4:8 layout
    assert [L.sharq_act_buffer_bytes(rows, K, 1, Pattern(4, 8, 1), w) for w in range(5)] == nv
    assert L.sharq_act_buffer_bytes(rows, K, 1, Pattern(3, 8, 1), 0) == 0   # odd n cannot be whole pairs
    assert L.sharq_weight_buffer_bytes(64, 128, 0, 0) == 64 * 64
    assert L.sharq_weight_buffer_bytes(64, 128, 1, 2) == 64 * 8


FAKE = 1 << 20   # never dereferenced: every case below is rejected (or empty) before any launch


def act(rows=8, K=128, n=2, m=4, fmt=0, off=0, pairs=0, mode=0, dn_meta=None, sp_dense=None):
    return Act(rows, K, fmt, Pattern(n, m, pairs), FAKE + off, FAKE, FAKE, FAKE, FAKE, None, mode, dn_meta, sp_dense)


@pytest.mark.parametrize("kw,M,K,ldx,nm,expect", [
    ({}, 8, 100, 128, (2, 4), EINVAL),        # K % 32
    ({}, 8, 128, 64, (2, 4), EINVAL),         # ldx < K
    ({}, -1, 128, 128, (2, 4), EINVAL),       # negative rows
    ({}, 8, 128, 128, (5, 4), EINVAL),        # n > m
    ({}, 8, 128, 128, (1, 4), EUNSUPPORTED),  # valid pattern, not built
    ({}, 8, 96, 96, (4, 8), EINVAL),          # K % m  (96 % 8 == 0 but mismatched act below) -> rows/K check
])
def test_prepare_rejects(L, kw, M, K, ldx, nm, expect):
    a = act(rows=M, K=K, n=nm[0], m=nm[1])
    if K == 96:
        a = act(rows=M, K=128, n=4, m=8)   # out->K disagrees with K
    st = L.sharq_prepare(FAKE, 0, M, K, ldx, None, 1e-6, Pattern(*nm), 0, None, ctypes.byref(a), None)
    assert st == expect


@pytest.mark.parametrize("nm,expect", [
    ((4, 8, 2), EINVAL),         # pairs must be 0 or 1
    ((3, 8, 1), EINVAL),         # odd n: not whole pairs
    ((2, 4, 1), EUNSUPPORTED),   # 2:4 in pairs (one pair of two) is valid but not built
    ((2, 8, 1), EUNSUPPORTED),
])
def test_prepare_pair_patterns(L, nm, expect):
    a = act(rows=8, K=128, n=nm[0], m=nm[1], pairs=nm[2])
    assert L.sharq_prepare(FAKE, 0, 8, 128, 128, None, 1e-6, Pattern(*nm), 0, None, ctypes.byref(a), None) == expect


def test_prepare_pairs_must_match_out(L):
    a = act(rows=8, K=128, n=4, m=8, pairs=0)
    assert L.sharq_prepare(FAKE, 0, 8, 128, 128, None, 1e-6, Pattern(4, 8, 1), 0, None, ctypes.byref(a),
                           None) == EINVAL
    empty = act(rows=0, K=128, n=4, m=8, pairs=1)
    assert L.sharq_prepare(FAKE, 0, 0, 128, 128, None, 1e-6, Pattern(4, 8, 1), 0, None, ctypes.byref(empty),
                           None) == OK


def test_prepare_residual_rejects(L):
    a = act()
    P = Pattern(2, 4, 0)
    call = lambda res, h, ldr, ldh, X=FAKE: L.sharq_prepare_residual(X, res, h, 0, 8, 128, 128, ldr, ldh, None, 1e-6,
                                                                     P, 0, None, ctypes.byref(a), None)
    assert call(None, FAKE, 128, 128) == EINVAL          # no residual
    assert call(FAKE, None, 128, 128) == EINVAL          # no h output
    assert call(FAKE, FAKE, 64, 128) == EINVAL           # ldr < K
    assert call(FAKE, FAKE, 128, 100) == EINVAL          # ldh < K
    assert call(FAKE + 2, FAKE, 128, 128) == EALIGN      # residual not 16-byte aligned
    assert call(FAKE, FAKE, 132, 128) == EALIGN          # residual row stride not 16 bytes
    assert call(FAKE, FAKE + 8, 128, 128) == EALIGN      # h not 16-byte aligned
    empty = act(rows=0)
    assert L.sharq_prepare_residual(FAKE, None, None, 0, 0, 128, 128, 128, 128, None, 1e-6, P, 0, None,
                                    ctypes.byref(empty), None) == OK


def test_prepare_null_and_alignment(L):
    a = act()
    assert L.sharq_prepare(None, 0, 8, 128, 128, None, 1e-6, Pattern(2, 4), 0, None, ctypes.byref(a), None) == EINVAL
    assert L.sharq_prepare(FAKE + 2, 0, 8, 128, 128, None, 1e-6, Pattern(2, 4), 0, None, ctypes.byref(a),
                           None) == EALIGN
    bad = act(off=8)   # sp_codes only 8-byte aligned
    assert L.sharq_prepare(FAKE, 0, 8, 128, 128, None, 1e-6, Pattern(2, 4), 0, None, ctypes.byref(bad),
                           None) == EALIGN
    assert L.sharq_prepare(FAKE, 2, 8, 128, 128, None, 1e-6, Pattern(2, 4), 0, None, ctypes.byref(a),
                           None) == EUNSUPPORTED   # fp32 X not built
    big = act(K=32768)
    assert L.sharq_prepare(FAKE, 0, 8, 32768, 32768, FAKE, 1e-6, Pattern(2, 4), 0, None, ctypes.byref(big),
                           None) == EUNSUPPORTED   # RMSNorm row longer than the register-resident maximum
    empty = act(rows=0)
    assert L.sharq_prepare(FAKE, 0, 0, 128, 128, None, 1e-6, Pattern(2, 4), 0, None, ctypes.byref(empty),
                           None) == OK             # nothing to do, nothing launched


def test_linear_rejects(L):
    a = act()
    w = Weight(64, 128, 1, 0, FAKE, FAKE, FAKE, None)
    assert L.sharq_linear(ctypes.byref(a), ctypes.byref(w), None, 2, 64, None) == EINVAL
    w_bad_k = Weight(64, 256, 1, 0, FAKE, FAKE, FAKE, None)
    assert L.sharq_linear(ctypes.byref(a), ctypes.byref(w_bad_k), FAKE, 2, 64, None) == EINVAL
    assert L.sharq_linear(ctypes.byref(a), ctypes.byref(w), FAKE, 2, 32, None) == EINVAL      # ldy < N
    assert L.sharq_linear(ctypes.byref(a), ctypes.byref(w), FAKE, 7, 64, None) == EUNSUPPORTED
    assert L.sharq_linear(ctypes.byref(a), ctypes.byref(w), FAKE + 2, 2, 64, None) == EALIGN   # fp32 Y
    w_nv = Weight(64, 128, 1, 1, FAKE, FAKE, FAKE, FAKE)
    assert L.sharq_linear(ctypes.byref(a), ctypes.byref(w_nv), FAKE, 2, 64, None) == EINVAL   # format mismatch
    empty = act(rows=0)
    assert L.sharq_linear(ctypes.byref(empty), ctypes.byref(w), FAKE, 2, 64, None) == OK


def test_grouped_rejects(L):
    a = act()
    w = Weight(64, 128, 4, 0, FAKE, FAKE, FAKE, None)
    assert L.sharq_linear_grouped(ctypes.byref(a), None, None, 8, ctypes.byref(w), FAKE, 2, 64, None) == EINVAL
    assert L.sharq_linear_grouped(ctypes.byref(a), None, FAKE, 9, ctypes.byref(w), FAKE, 2, 64, None) == EINVAL
    assert L.sharq_linear_grouped(ctypes.byref(a), FAKE + 1, FAKE, 8, ctypes.byref(w), FAKE, 2, 64,
                                  None) == EALIGN
    w_many = Weight(64, 128, 5000, 0, FAKE, FAKE, FAKE, None)
    assert L.sharq_linear_grouped(ctypes.byref(a), None, FAKE, 8, ctypes.byref(w_many), FAKE, 2, 64,
                                  None) == EINVAL
    assert L.sharq_linear_grouped(ctypes.byref(a), None, FAKE, 0, ctypes.byref(w), FAKE, 2, 64, None) == OK


def test_quantize_weight_rejects(L):
    w = Weight(64, 128, 1, 0, FAKE, FAKE, FAKE, None)
    assert L.sharq_quantize_weight(None, 0, 64, 128, 128, ctypes.byref(w), None) == EINVAL
    assert L.sharq_quantize_weight(FAKE, 0, 64, 100, 128, ctypes.byref(w), None) == EINVAL
    assert L.sharq_quantize_weight(FAKE, 0, 32, 128, 128, ctypes.byref(w), None) == EINVAL   # out->N mismatch
    assert L.sharq_quantize_weight(FAKE, 1, 64, 128, 128, ctypes.byref(w), None) == EUNSUPPORTED
    assert L.sharq_quantize_weight(FAKE, 0, 64, 128, 132, ctypes.byref(w), None) == EALIGN
    w0 = Weight(0, 128, 1, 0, FAKE, FAKE, FAKE, None)
    assert L.sharq_quantize_weight(FAKE, 0, 0, 128, 128, ctypes.byref(w0), None) == OK


def nv_act(rows=8, K=128, ts=FAKE):
    return Act(rows, K, 1, Pattern(2, 4), FAKE, FAKE, FAKE, FAKE, FAKE, ts)


def test_nvfp4_needs_tensor_scales(L):
    w = Weight(64, 128, 1, 1, FAKE, FAKE, FAKE, FAKE)
    no_ts = nv_act(ts=None)
    assert L.sharq_linear(ctypes.byref(no_ts), ctypes.byref(w), FAKE, 2, 64, None) == EINVAL
    w_no_ts = Weight(64, 128, 1, 1, FAKE, FAKE, FAKE, None)
    assert L.sharq_linear(ctypes.byref(nv_act()), ctypes.byref(w_no_ts), FAKE, 2, 64, None) == EINVAL
    w_no_dn = Weight(64, 128, 1, 1, FAKE, FAKE, None, FAKE)
    assert L.sharq_linear(ctypes.byref(nv_act()), ctypes.byref(w_no_dn), FAKE, 2, 64, None) == EINVAL
    assert L.sharq_linear(ctypes.byref(nv_act(ts=FAKE + 2)), ctypes.byref(w), FAKE, 2, 64, None) == EALIGN
    assert L.sharq_quantize_weight(FAKE, 0, 64, 128, 128, ctypes.byref(w_no_ts), None) == EINVAL
    assert L.sharq_prepare(FAKE, 0, 8, 128, 128, None, 1e-6, Pattern(2, 4), 1, None, ctypes.byref(no_ts),
                           None) == EINVAL
    assert L.sharq_prepare(FAKE, 0, 8, 128, 128, None, 1e-6, Pattern(2, 4), 1, FAKE + 1, ctypes.byref(nv_act()),
                           None) == EALIGN
    # the activation's format must be the one asked for
    assert L.sharq_prepare(FAKE, 0, 8, 128, 128, None, 1e-6, Pattern(2, 4), 0, None, ctypes.byref(nv_act()),
                           None) == EINVAL


def test_nvfp4_grouped_not_built(L):
    w = Weight(64, 128, 4, 1, FAKE, FAKE, FAKE, FAKE)
    assert L.sharq_linear_grouped(ctypes.byref(nv_act()), None, FAKE, 8, ctypes.byref(w), FAKE, 2, 64,
                                  None) == EUNSUPPORTED


# ----------------------------------------------------------------------------- path combinations

SHARQ, SPARSE, DENSE, DENSE_DENSE, SPARSE_SPARSE = range(5)


def test_buffer_sizes_per_mode(L):
    rows, K = 5, 256
    f = lambda fmt, nm, mode: [L.sharq_act_buffer_bytes_mode(rows, K, fmt, nm, mode, w) for w in range(6)]
    p24 = Pattern(2, 4)
    # which: 0 sp_codes, 1 sp_meta, 2 sp_scale, 3 dn_codes, 4 dn_scale, 5 dn_meta
    assert f(0, p24, SHARQ) == [rows * K // 4, rows * K // 8, rows * K // 32, rows * K // 2, rows * K // 32, 0]
    assert f(0, p24, SHARQ)[:5] == [L.sharq_act_buffer_bytes(rows, K, 0, p24, w) for w in range(5)]
    assert f(0, p24, SPARSE) == [rows * K // 4, rows * K // 8, rows * K // 32, 0, 0, 0]
    assert f(1, p24, DENSE) == [0, 0, 0, rows * K // 2, rows * K // 16, 0]
    assert f(1, p24, DENSE_DENSE) == [rows * K // 2, 0, rows * K // 16, rows * K // 2, rows * K // 16, 0]
    assert f(1, Pattern(4, 8, 1), SPARSE_SPARSE) == [rows * K // 4, rows * K // 8, rows * K // 32,
                                                     rows * K // 4, rows * K // 32, rows * K // 8]
    # a dense-only mode accepts a valid pattern that no sparse path is built for
    assert f(0, Pattern(1, 4), DENSE)[3] == rows * K // 2
    assert f(0, Pattern(1, 4), SPARSE) == [0] * 6
    assert f(0, p24, 5) == [0] * 6 and f(0, p24, -1) == [0] * 6


def test_mode_rejections(L):
    def prep(a, nm=(2, 4)):
        return L.sharq_prepare(FAKE, 0, a.rows, a.K, a.K, None, 1e-6, Pattern(*nm), a.fmt, None, ctypes.byref(a),
                               None)
    assert prep(act(mode=5)) == EINVAL
    assert prep(act(mode=-1)) == EINVAL
    assert prep(act(n=1, m=4, mode=SPARSE), (1, 4)) == EUNSUPPORTED
    assert prep(act(n=1, m=4, mode=SPARSE_SPARSE), (1, 4)) == EUNSUPPORTED
    assert prep(act(mode=SPARSE_SPARSE, dn_meta=None)) == EINVAL        # a sparse path 2 needs its metadata
    assert prep(act(mode=SPARSE_SPARSE, dn_meta=FAKE + 2)) == EALIGN
    # the fused residual add and the grouped GEMM are built for the method only
    a = act(mode=DENSE_DENSE)
    st = L.sharq_prepare_residual(FAKE, FAKE, FAKE, 0, 8, 128, 128, 128, 128, None, 1e-6, Pattern(2, 4), 0, None,
                                  ctypes.byref(a), None)
    assert st == EUNSUPPORTED
    w = Weight(64, 128, 1, 0, FAKE, FAKE, FAKE, None)
    st = L.sharq_linear_grouped(ctypes.byref(act(mode=SPARSE)), None, FAKE, 8, ctypes.byref(w), FAKE, 0, 64, None)
    assert st == EUNSUPPORTED


def test_mode_empty_calls_launch_nothing(L):
    for mode in range(5):
        a = act(rows=0, mode=mode)
        assert L.sharq_prepare(None, 0, 0, 128, 128, None, 1e-6, Pattern(2, 4), 0, None, ctypes.byref(a), None) == OK
        w = Weight(64, 128, 1, 0, FAKE, FAKE, FAKE, None)
        assert L.sharq_linear(ctypes.byref(a), ctypes.byref(w), None, 0, 64, None) == OK


# ----------------------------------------------------------------------------- HiF4

HIF4 = 2


def test_hif4_buffer_sizes(L):
    rows, K = 3, 256
    got = [L.sharq_act_buffer_bytes(rows, K, HIF4, Pattern(2, 4), w) for w in range(5)]
    assert got == [rows * K // 4, rows * K // 8, rows * K // 16, rows * K // 2, rows * K // 16]
    assert L.sharq_act_buffer_bytes(rows, 96, HIF4, Pattern(2, 4), 3) == 0          # K % 64
    assert [L.sharq_weight_buffer_bytes(40, K, HIF4, w) for w in range(3)] == [40 * K // 2, 40 * K // 16, 40 * K // 16]


def test_hif4_rejections(L):
    def prep(a, nm=(2, 4), K=None):
        K = K or a.K
        return L.sharq_prepare(FAKE, 0, a.rows, K, K, None, 1e-6, Pattern(*nm), HIF4, None, ctypes.byref(a), None)
    assert prep(act(K=96, fmt=HIF4)) == EINVAL                             # K not a multiple of 64
    assert prep(act(n=4, m=8, fmt=HIF4), (4, 8)) == EUNSUPPORTED           # built with 2:4 only
    assert prep(act(fmt=HIF4, mode=SPARSE)) == EUNSUPPORTED                # the method's combination only
    a = act(fmt=HIF4)
    st = L.sharq_prepare_residual(FAKE, FAKE, FAKE, 0, 8, 128, 128, 128, 128, None, 1e-6, Pattern(2, 4), HIF4, None,
                                  ctypes.byref(a), None)
    assert st == EUNSUPPORTED
    w = Weight(64, 128, 1, HIF4, FAKE, FAKE, FAKE, None)
    st = L.sharq_linear_grouped(ctypes.byref(act(fmt=HIF4)), None, FAKE, 8, ctypes.byref(w), FAKE, 0, 64, None)
    assert st == EUNSUPPORTED
    wq = Weight(64, 96, 1, HIF4, FAKE, FAKE, FAKE, None)
    assert L.sharq_quantize_weight(FAKE, 0, 64, 96, 96, ctypes.byref(wq), None) == EINVAL
    # formats must agree between activation and weight
    wmx = Weight(64, 128, 1, 0, FAKE, FAKE, FAKE, None)
    assert L.sharq_linear(ctypes.byref(act(fmt=HIF4)), ctypes.byref(wmx), FAKE, 0, 64, None) == EINVAL


def test_silu_mul_rejections(L):
    L.sharq_prepare_silu_mul.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int,
                                         ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                         ctypes.c_int64, Pattern, ctypes.c_int, ctypes.c_void_p, ctypes.POINTER(Act),
                                         ctypes.c_void_p]

    def call(a, up=FAKE, h=None, ldu=128, ldh=128, fmt=0):
        return L.sharq_prepare_silu_mul(FAKE, up, h, 0, a.rows, a.K, a.K, ldu, ldh, Pattern(a.nm.n, a.nm.m),
                                        fmt, None, ctypes.byref(a), None)
    assert call(act(), up=None) == EINVAL
    assert call(act(), ldu=64) == EINVAL
    assert call(act(), h=FAKE, ldh=64) == EINVAL
    assert call(act(), h=FAKE + 8) == EALIGN
    assert call(act(mode=DENSE)) == EUNSUPPORTED
    assert call(act(fmt=HIF4), fmt=HIF4) == EUNSUPPORTED
    assert call(act(rows=0), up=None) == OK


def test_dense_backbone_copy_rejections(L):
    def prep(a, fmt=0):
        return L.sharq_prepare(FAKE, 0, a.rows, a.K, a.K, None, 1e-6, Pattern(a.nm.n, a.nm.m), fmt, None,
                               ctypes.byref(a), None)
    assert prep(act(sp_dense=FAKE + 8)) == EALIGN
    assert prep(act(fmt=2, sp_dense=FAKE), fmt=2) == EUNSUPPORTED       # MXFP4 and NVFP4, not HiF4
    nv = Act(8, 160, 1, Pattern(2, 4, 0), None, None, FAKE, FAKE, FAKE, FAKE, 0, None, FAKE)
    assert L.sharq_prepare(FAKE, 0, 8, 160, 160, None, 1e-6, Pattern(2, 4), 1, None, ctypes.byref(nv),
                           None) == EUNSUPPORTED                        # NVFP4 dense-only: K a multiple of 128
    nv = act(fmt=1, sp_dense=FAKE + 8)
    nv.tensor_scale = FAKE
    assert prep(nv, fmt=1) == EALIGN
    assert prep(act(mode=SPARSE, sp_dense=FAKE)) == EUNSUPPORTED        # the method's combination only


def test_scale_rule_debug_and_dense_only_rejections(L):
    """The E8M0 rule, the debug outputs and the dense-only backbone are
    validated before any launch."""
    def prep(a, K=128, fmt=0, nm=(2, 4, 0)):
        return L.sharq_prepare(FAKE, 0, a.rows, K, K, None, ctypes.c_float(1e-6), Pattern(*nm), fmt, None,
                               ctypes.byref(a), None)
    a = act()
    a.scale_rule = 2
    assert prep(a) == EINVAL
    nv = act(fmt=1)
    nv.tensor_scale = FAKE
    nv.scale_rule = 1
    assert prep(nv, fmt=1) == EUNSUPPORTED            # the ceil rule is an MXFP4 option
    m = act(mode=1)
    m.scale_rule = 1
    assert prep(m) == EUNSUPPORTED                    # ... of the method's own combination
    h = act(fmt=2)
    h.dbg_mask = FAKE
    assert prep(h, fmt=2) == EUNSUPPORTED             # no debug outputs for HiF4
    d = act()
    d.dbg_r = FAKE + 2
    assert prep(d) == EALIGN
    # dense-only backbone: sp_codes and sp_meta NULL beside sp_dense
    do = Act(8, 160, 0, Pattern(2, 4, 0), None, None, FAKE, FAKE, FAKE, None, 0, None, FAKE)
    assert prep(do, K=160) == EUNSUPPORTED            # K must be a multiple of 128
    half = Act(8, 128, 0, Pattern(2, 4, 0), FAKE, None, FAKE, FAKE, FAKE, None, 0, None, FAKE)
    assert prep(half) == EINVAL                       # codes without metadata
    w = Weight(64, 128, 1, 1, FAKE, FAKE, FAKE, FAKE, 1)
    assert L.sharq_quantize_weight(FAKE, 0, 64, 128, 128, ctypes.byref(w), None) == EUNSUPPORTED
    w = Weight(64, 128, 1, 0, FAKE, FAKE, FAKE, None, 7)
    assert L.sharq_quantize_weight(FAKE, 0, 64, 128, 128, ctypes.byref(w), None) == EINVAL


PROBE_LIB = os.path.join(ROOT, "paper_2606_26587_amd", "libsharq_probe.so")
PROBE_HEADER = os.path.join(ROOT, "include", "sharq_probe.h")


@pytest.mark.skipif(not os.path.exists(PROBE_LIB), reason="libsharq_probe.so not built")
def test_probe_library_exports_and_rejects():
    """The benchmark's MFMA-rate probe library exports what its header
    declares and rejects bad arguments before any launch."""
    names = re.findall(r"\bint\s+(sharq_probe_\w+)\s*\(", open(PROBE_HEADER).read())
    assert names == ["sharq_probe_mfma_fp4", "sharq_probe_mfma_bf16", "sharq_probe_mfma_f16"]
    P = ctypes.CDLL(PROBE_LIB)
    fake = 1 << 20   # never dereferenced
    hip_invalid_value = 1
    for n in names:
        assert hasattr(P, n), n
        fn = getattr(P, n)
        fn.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        for iters, wgs, sink, clk in [(0, 1, fake, fake), (1, 0, fake, fake), (1, 1, None, fake), (1, 1, fake, None)]:
            assert fn(iters, wgs, sink, clk, None) == hip_invalid_value, n
