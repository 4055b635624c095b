"""The plain C oracle (oracle/sharq_ref.c) against the NumPy oracle: two
independent implementations of the same definitions and readings must agree
byte for byte on every prepared buffer, the keep mask and r, and on the weight
bytes; their fp64 GEMMs agree to rounding (exactly on exact-sum operands).
MXFP4 and NVFP4 (with the per-tensor scale's bits, and E4M3 rounding against
an exhaustive search).
Also: the C oracle's argument checks return the library's status codes for
the arguments both validate, and its OpenMP rows do not change results."""

import ctypes
import os

import numpy as np
import pytest

from oracle import build_ref
from oracle import sharq_oracle as O
from paper_2606_26587_amd import synth


@pytest.fixture(scope="module")
def C():
    return build_ref.load()


def ptr(a):
    return None if a is None else ctypes.c_void_p(a.ctypes.data)


def c_prepare(C, x, g, eps, n, m, rule=0):
    T, K = x.shape
    out = {"sp_codes": np.zeros((T, K * n // m // 2), np.uint8), "sp_meta": np.zeros((T, K // 8), np.uint8),
           "sp_scale": np.zeros((T, K // 32), np.uint8), "dn_codes": np.zeros((T, K // 2), np.uint8),
           "dn_scale": np.zeros((T, K // 32), np.uint8), "r": np.zeros(T, np.float32),
           "keep": np.zeros((T, K // 8), np.uint8)}
    x = np.ascontiguousarray(x)
    st = C.sharq_ref_prepare(ptr(x), T, K, K, ptr(g), ctypes.c_float(eps), n, m, rule, *(ptr(out[k]) for k in (
        "sp_codes", "sp_meta", "sp_scale", "dn_codes", "dn_scale", "r", "keep")))
    assert st == 0, st
    return out


def special(kind, T, K, seed):
    rng = np.random.default_rng(seed)
    if kind == "zeros":
        x = np.zeros((T, K), np.float32)
        x[:, ::3] = -0.0
    elif kind == "ties":
        x = rng.integers(-3, 4, size=(T, K)).astype(np.float32)
    elif kind == "subnormal":
        x = (rng.standard_normal((T, K)) * 1e-39).astype(np.float32)
        x[:, ::5] *= 1e-2
    elif kind == "huge":
        x = (rng.standard_normal((T, K)) * 1e30).astype(np.float32)
    else:
        x = rng.standard_normal((T, K)).astype(np.float32)
        x[0] = 0.0
        x[1, ::2] = 1e-40
        x[2] *= 1e25
        x[3, 5::7] = 6000.0
    return synth.f32_to_bf16_bits(x)


CASES = [(8, 128, True, 2, 4, "floor"), (37, 416, True, 2, 4, "floor"), (37, 416, False, 4, 8, "floor"),
         (9, 4096, True, 2, 4, "ceil"), (5, 14336, False, 2, 4, "floor"), (12, 768, True, 4, 8, "ceil"),
         (3, 96, True, 2, 4, "floor")]


@pytest.mark.parametrize("T,K,use_gamma,n,m,rule", CASES)
def test_c_prepare_equals_numpy(C, T, K, use_gamma, n, m, rule):
    x = synth.activations(T, K, seed=T * K)
    g = synth.gamma(K, seed=K) if use_gamma else None
    c = c_prepare(C, x, g, 1e-5, n, m, 1 if rule == "ceil" else 0)
    o = O.prepare(x, g, 1e-5, n, m, "mx", scale_rule=rule)
    for k in O.ACT_BUFFERS:
        assert np.array_equal(c[k], o[k]), k
    assert np.array_equal(c["keep"], np.packbits(o["keep"].astype(np.uint8), axis=1, bitorder="little"))
    assert np.array_equal(c["r"].view(np.uint32), np.asarray(o["r"], np.float32).view(np.uint32))


@pytest.mark.parametrize("kind", ["zeros", "ties", "subnormal", "huge", "mixed"])
@pytest.mark.parametrize("n,m", [(2, 4), (4, 8)])
@pytest.mark.parametrize("use_gamma", [True, False])
def test_c_prepare_edge_values(C, kind, n, m, use_gamma):
    x = special(kind, 12, 256, seed=len(kind))
    g = synth.gamma(256, seed=3) if use_gamma else None
    c = c_prepare(C, x, g, 1e-6, n, m)
    with np.errstate(over="ignore"):
        o = O.prepare(x, g, 1e-6, n, m, "mx")
    for k in O.ACT_BUFFERS:
        assert np.array_equal(c[k], o[k]), (kind, k)


@pytest.mark.parametrize("rule", ["floor", "ceil"])
def test_c_weight_equals_numpy(C, rule):
    N, K = 70, 640
    w = np.ascontiguousarray(synth.weight(N, K, seed=5))
    codes, scale = np.zeros((N, K // 2), np.uint8), np.zeros((N, K // 32), np.uint8)
    assert C.sharq_ref_quantize_weight(ptr(w), N, K, K, 1 if rule == "ceil" else 0, ptr(codes), ptr(scale)) == 0
    o = O.quantize_weight(w, "mx", scale_rule=rule)
    assert np.array_equal(codes, o["codes"]) and np.array_equal(scale, o["scale"])


def c_linear(C, o, wq, n, m):
    T, K, N = o["rows"], o["K"], wq["N"]
    Y = np.zeros((T, N), np.float64)
    args = [np.ascontiguousarray(o[k]) for k in ("sp_codes", "sp_meta", "sp_scale", "dn_codes", "dn_scale")]
    assert C.sharq_ref_linear(T, K, n, m, *(ptr(a) for a in args), N, ptr(np.ascontiguousarray(wq["codes"])),
                              ptr(np.ascontiguousarray(wq["scale"])), ptr(Y), N) == 0
    return Y


@pytest.mark.parametrize("T,N,K,n,m", [(8, 64, 128, 2, 4), (33, 100, 1024, 4, 8), (5, 40, 4096, 2, 4)])
def test_c_linear_agrees_with_numpy(C, T, N, K, n, m):
    x = synth.activations(T, K, seed=N)
    o = O.prepare(x, synth.gamma(K, seed=2), 1e-6, n, m, "mx")
    wq = O.quantize_weight(synth.weight(N, K, seed=T), "mx")
    y_c, y_o = c_linear(C, o, wq, n, m), O.linear(o, wq)
    den = O.linear_abs(o, wq)
    assert np.max(np.abs(y_c - y_o) / np.where(den > 0, den, 1.0)) <= 1e-13


def test_c_linear_exact_on_exact_sums(C):
    """Unit scales and codes: every sum is exact in fp64, so the two
    implementations (loop order and BLAS order) give identical results."""
    rng = np.random.default_rng(9)
    T, N, K = 6, 30, 512
    keep = np.zeros((T, K), bool)
    for t in range(T):
        for g in range(K // 4):
            keep[t, 4 * g + rng.choice(4, 2, replace=False)] = True
    sp = np.where(keep, rng.integers(0, 16, (T, K)), 0).astype(np.uint8)
    spc, spm = O.pack_backbone(sp, keep, 2, 4)
    o = {"rows": T, "K": K, "n": 2, "m": 4, "fmt": "mx", "tensor_scale": None, "mode": "sharq",
         "sp_codes": spc, "sp_meta": spm, "sp_scale": np.full((T, K // 32), 127, np.uint8),
         "dn_codes": O.pack_nibbles(rng.integers(0, 16, (T, K)).astype(np.uint8)),
         "dn_scale": np.full((T, K // 32), 127, np.uint8)}
    wq = {"N": N, "K": K, "fmt": "mx", "tensor_scale": None,
          "codes": O.pack_nibbles(rng.integers(0, 16, (N, K)).astype(np.uint8)),
          "scale": np.full((N, K // 32), 127, np.uint8)}
    wq["scale_dn"] = wq["scale"]
    assert np.array_equal(c_linear(C, o, wq, 2, 4), O.linear(o, wq))


def test_c_threads_do_not_change_results(C):
    x = synth.activations(40, 2048, seed=4)
    g = synth.gamma(2048, seed=4)
    outs = []
    for th in (1, 3, 0):
        C.sharq_ref_set_threads(th)
        outs.append(c_prepare(C, x, g, 1e-5, 2, 4))
    C.sharq_ref_set_threads(0)
    for k in O.ACT_BUFFERS:
        assert np.array_equal(outs[0][k], outs[1][k]) and np.array_equal(outs[0][k], outs[2][k])


# --------------------------------------------------------------------------- NVFP4

NV_BUFS = ("sp_codes", "sp_meta", "sp_scale", "dn_codes", "dn_scale")


def c_prepare_nv(C, x, g, eps, n, m, pairs=False, ts=None):
    T, K = x.shape
    out = {"sp_codes": np.zeros((T, K * n // m // 2), np.uint8), "sp_meta": np.zeros((T, K // 8), np.uint8),
           "sp_scale": np.zeros((T, K // 32), np.uint8), "dn_codes": np.zeros((T, K // 2), np.uint8),
           "dn_scale": np.zeros((T, K // 16), np.uint8)}
    tso = np.zeros(1, np.float32)
    tsi = None if ts is None else np.array([ts], np.float32)
    x = np.ascontiguousarray(x)
    st = C.sharq_ref_prepare_nv(ptr(x), T, K, K, ptr(g), eps, n, m, int(pairs), ptr(tsi), ptr(tso),
                                *(ptr(out[k]) for k in NV_BUFS))
    assert st == 0, st
    out["tensor_scale"] = tso[0]
    return out


def assert_nv_prep_equal(c, o, tag):
    for k in NV_BUFS:
        assert np.array_equal(c[k], o[k]), (tag, k)
    assert np.float32(c["tensor_scale"]).view(np.uint32) == np.float32(o["tensor_scale"]).view(np.uint32), tag


NV_CASES = [(8, 128, True, 2, 4, False, None), (37, 416, True, 2, 4, False, None),
            (37, 416, False, 4, 8, False, None), (20, 1024, True, 4, 8, True, None),
            (9, 3584, True, 2, 4, False, None), (5, 18944, False, 2, 4, False, None),
            (12, 768, True, 4, 8, True, 0.02), (3, 96, True, 2, 4, False, 3e-4)]


@pytest.mark.parametrize("T,K,use_gamma,n,m,pairs,ts", NV_CASES)
def test_c_prepare_nv_equals_numpy(C, T, K, use_gamma, n, m, pairs, ts):
    """NVFP4 preparation (per-tensor scale computed or given, 2:4, 4:8, 4:8
    in pairs): every buffer and the per-tensor scale's bits."""
    x = synth.activations(T, K, seed=T + K)
    g = synth.gamma(K, seed=K + 2) if use_gamma else None
    c = c_prepare_nv(C, x, g, 1e-6, n, m, pairs, ts)
    o = O.prepare(x, g, 1e-6, n, m, "nv", tensor_scale=ts, pairs=pairs)
    assert_nv_prep_equal(c, o, f"T{T}K{K}")


@pytest.mark.parametrize("kind", ["zeros", "ties", "subnormal", "huge", "mixed"])
@pytest.mark.parametrize("n,m,pairs", [(2, 4, False), (4, 8, False), (4, 8, True)])
@pytest.mark.parametrize("use_gamma", [True, False])
def test_c_prepare_nv_edge_values(C, kind, n, m, pairs, use_gamma):
    """All-zero input (S = 1, every block scale 0, signed-zero codes), ties,
    subnormals, huge values and mixed rows whose block scales underflow."""
    x = special(kind, 12, 256, seed=len(kind) + 7)
    g = synth.gamma(256, seed=5) if use_gamma else None
    c = c_prepare_nv(C, x, g, 1e-6, n, m, pairs)
    with np.errstate(over="ignore", under="ignore"):
        o = O.prepare(x, g, 1e-6, n, m, "nv", pairs=pairs)
    assert_nv_prep_equal(c, o, kind)


@pytest.mark.parametrize("N,K", [(70, 640), (33, 18944), (5, 96)])
def test_c_weight_nv_equals_numpy(C, N, K):
    w = np.ascontiguousarray(synth.weight(N, K, seed=N + K))
    codes, scale = np.zeros((N, K // 2), np.uint8), np.zeros((N, K // 32), np.uint8)
    ts = np.zeros(1, np.float32)
    assert C.sharq_ref_quantize_weight_nv(ptr(w), N, K, K, ptr(codes), ptr(scale), ptr(ts)) == 0
    o = O.quantize_weight(w, "nv")
    assert np.array_equal(codes, o["codes"]) and np.array_equal(scale, o["scale"])
    assert ts.view(np.uint32)[0] == np.float32(o["tensor_scale"]).view(np.uint32)


def c_linear_nv(C, o, wq, n, m):
    T, K, N = o["rows"], o["K"], wq["N"]
    Y = np.zeros((T, N), np.float64)
    args = [np.ascontiguousarray(o[k]) for k in NV_BUFS]
    assert C.sharq_ref_linear_nv(T, K, n, m, *(ptr(a) for a in args), float(o["tensor_scale"]), N,
                                 ptr(np.ascontiguousarray(wq["codes"])), ptr(np.ascontiguousarray(wq["scale"])),
                                 float(wq["tensor_scale"]), ptr(Y), N) == 0
    return Y


@pytest.mark.parametrize("T,N,K,n,m,pairs", [(8, 64, 128, 2, 4, False), (33, 100, 1024, 4, 8, True),
                                             (5, 40, 3584, 2, 4, False)])
def test_c_linear_nv_agrees_with_numpy(C, T, N, K, n, m, pairs):
    x = synth.activations(T, K, seed=N + 1)
    o = O.prepare(x, synth.gamma(K, seed=4), 1e-6, n, m, "nv", pairs=pairs)
    wq = O.quantize_weight(synth.weight(N, K, seed=T + 1), "nv")
    y_c, y_o = c_linear_nv(C, o, wq, n, m), O.linear(o, wq)
    den = O.linear_abs(o, wq)
    assert np.max(np.abs(y_c - y_o) / np.where(den > 0, den, 1.0)) <= 1e-13


def test_c_linear_nv_exact_on_exact_sums(C):
    """Unit block and tensor scales: every sum is exact in fp64, so the two
    implementations give identical results; then the same operands with the
    tensor scales 2^-3 and 2^5, which scale every output exactly."""
    rng = np.random.default_rng(11)
    T, N, K = 6, 30, 512
    keep = np.zeros((T, K), bool)
    for t in range(T):
        for g in range(K // 8):
            keep[t, 8 * g + rng.choice(8, 4, replace=False)] = True
    sp = np.where(keep, rng.integers(0, 16, (T, K)), 0).astype(np.uint8)
    spc, spm = O.pack_backbone(sp, keep, 4, 8)
    one = 0x38   # E4M3 1.0
    o = {"rows": T, "K": K, "n": 4, "m": 8, "fmt": "nv", "tensor_scale": np.float32(1.0), "mode": "sharq",
         "sp_codes": spc, "sp_meta": spm, "sp_scale": np.full((T, K // 32), one, np.uint8),
         "dn_codes": O.pack_nibbles(rng.integers(0, 16, (T, K)).astype(np.uint8)),
         "dn_scale": np.full((T, K // 16), one, np.uint8)}
    ws = np.full((N, K // 32), one, np.uint8)
    wq = {"N": N, "K": K, "fmt": "nv", "tensor_scale": np.float32(1.0),
          "codes": O.pack_nibbles(rng.integers(0, 16, (N, K)).astype(np.uint8)), "scale": ws,
          "scale_dn": np.repeat(ws, 2, axis=1)}
    y1 = c_linear_nv(C, o, wq, 4, 8)
    assert np.array_equal(y1, O.linear(o, wq))
    o["tensor_scale"], wq["tensor_scale"] = np.float32(2.0 ** -3), np.float32(2.0 ** 5)
    assert np.array_equal(c_linear_nv(C, o, wq, 4, 8), y1 * 4.0)
    assert np.array_equal(O.linear(o, wq), y1 * 4.0)


def test_e4m3_rounding_numpy_equals_exhaustive_search(C):
    """The NumPy oracle's E4M3 rounding (binade arithmetic) against the format's
    definition, nearest of the 126 finite non-negative values with ties to the
    even code and saturation at 448, found by exhaustive search in C: every
    value, every midpoint between neighbours and the floats next to each
    midpoint, the subnormal range, zero, and values past 448."""
    vals = O.e4m3_values()
    mids = (vals[:-1] + vals[1:]) / 2.0
    probe = [np.float32(0.0), np.float32(2.0 ** -11), np.float32(2.0 ** -10), np.float32(500.0),
             np.float32(464.0), np.float32(3.0e38)]
    for v in np.concatenate([vals, mids]).astype(np.float32):
        probe += [v, np.nextafter(v, np.float32(0.0)), np.nextafter(v, np.float32(np.inf))]
    rng = np.random.default_rng(3)
    probe += list((2.0 ** rng.uniform(-12, 10, 4000)).astype(np.float32))
    a = np.array(probe, np.float32)
    want = O.e4m3_encode_bits(O.e4m3_round(a))
    got = np.array([C.sharq_ref_e4m3_code(float(v)) for v in a], np.uint8)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(float(a[i]), int(got[i]), int(want[i])) for i in bad[:5]]
    # the exhaustive search is the definition: spot values
    assert C.sharq_ref_e4m3_code(448.0) == 0x7E and C.sharq_ref_e4m3_code(1.0) == 0x38
    assert C.sharq_ref_e4m3_code(2.0 ** -9) == 0x01 and C.sharq_ref_e4m3_code(2.0 ** -10) == 0x00


LIB = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2606_26587_amd",
                   "libsharq.so")


@pytest.mark.skipif(not os.path.exists(LIB), reason="libsharq.so not built")
def test_c_status_codes_match_the_library(C):
    """For the arguments both validate, the C oracle rejects what the library
    rejects, with the same status (the library's checks run before any
    launch, so no GPU is involved)."""
    class Pattern(ctypes.Structure):
        _fields_ = [("n", ctypes.c_int32), ("m", ctypes.c_int32), ("pairs", ctypes.c_int32)]

    class Act(ctypes.Structure):
        _fields_ = [("rows", ctypes.c_int64), ("K", ctypes.c_int64), ("fmt", ctypes.c_int), ("nm", Pattern),
                    ("sp_codes", ctypes.c_void_p), ("sp_meta", ctypes.c_void_p), ("sp_scale", ctypes.c_void_p),
                    ("dn_codes", ctypes.c_void_p), ("dn_scale", ctypes.c_void_p), ("tensor_scale", ctypes.c_void_p),
                    ("mode", ctypes.c_int), ("dn_meta", ctypes.c_void_p), ("sp_dense", ctypes.c_void_p),
                    ("scale_rule", ctypes.c_int), ("dbg_mask", ctypes.c_void_p), ("dbg_r", ctypes.c_void_p)]

    L = ctypes.CDLL(LIB)
    L.sharq_prepare.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                ctypes.c_void_p, ctypes.c_float, Pattern, ctypes.c_int, ctypes.c_void_p,
                                ctypes.POINTER(Act), ctypes.c_void_p]
    fake = 1 << 20   # never dereferenced: every case is rejected before any work
    cases = [  # (M, K, ldx, n, m, rule, eps)
        (8, 100, 128, 2, 4, 0, 1e-6),    # K % 32
        (8, 128, 64, 2, 4, 0, 1e-6),     # ldx < K
        (-1, 128, 128, 2, 4, 0, 1e-6),   # negative rows
        (8, 128, 128, 5, 4, 0, 1e-6),    # n > m
        (8, 128, 128, 1, 4, 0, 1e-6),    # a valid pattern that is not built
        (8, 128, 128, 2, 4, 3, 1e-6),    # no such E8M0 rule
        (8, 128, 128, 2, 4, 0, -1.0),    # negative eps
    ]
    for M, K, ldx, n, m, rule, eps in cases:
        a = Act(M, K, 0, Pattern(n, m, 0), fake, fake, fake, fake, fake, None, 0, None, None, rule)
        lib = L.sharq_prepare(fake, 0, M, K, ldx, fake, ctypes.c_float(eps), Pattern(n, m, 0), 0, None,
                              ctypes.byref(a), None)
        ref = C.sharq_ref_prepare(ctypes.c_void_p(fake), M, K, ldx, ctypes.c_void_p(fake), ctypes.c_float(eps), n,
                                  m, rule, *([ctypes.c_void_p(fake)] * 5), None, None)
        assert lib == ref != 0, (M, K, ldx, n, m, rule, eps, lib, ref)
