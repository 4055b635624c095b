"""Build the plain C oracle (oracle/sharq_ref.c) as oracle/libsharq_ref.so.

Test infrastructure: only tests, the package's smoke check and the benchmark's
CPU-baseline leg load the result.  Compiled with gcc, IEEE arithmetic (no
contraction into fused multiply-add, no fast-math) and OpenMP over rows.

    python -m oracle.build_ref
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "sharq_ref.c")
LIB = os.path.join(HERE, "libsharq_ref.so")

FLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-ffp-contract=off", "-fno-fast-math",
         "-fexcess-precision=standard"]


def build(verbose: bool = True) -> str:
    cc = os.environ.get("CC", shutil.which("gcc") or "gcc")
    tmp = LIB + ".tmp"
    cmd = [cc, *FLAGS, SRC, "-o", tmp, "-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"building the C oracle failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    return LIB


def load():
    """ctypes handle of the C oracle (built on first use)."""
    import ctypes
    if not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        build(verbose=False)
    L = ctypes.CDLL(LIB)
    vp, i64 = ctypes.c_void_p, ctypes.c_int64
    L.sharq_ref_prepare.argtypes = [vp, i64, i64, i64, vp, ctypes.c_float, ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                    vp, vp, vp, vp, vp, vp, vp]
    L.sharq_ref_prepare.restype = ctypes.c_int
    L.sharq_ref_quantize_weight.argtypes = [vp, i64, i64, i64, ctypes.c_int, vp, vp]
    L.sharq_ref_quantize_weight.restype = ctypes.c_int
    L.sharq_ref_linear.argtypes = [i64, i64, ctypes.c_int, ctypes.c_int, vp, vp, vp, vp, vp, i64, vp, vp, vp, i64]
    L.sharq_ref_linear.restype = ctypes.c_int
    f32, i32 = ctypes.c_float, ctypes.c_int
    L.sharq_ref_prepare_nv.argtypes = [vp, i64, i64, i64, vp, f32, i32, i32, i32, vp, vp, vp, vp, vp, vp, vp]
    L.sharq_ref_prepare_nv.restype = ctypes.c_int
    L.sharq_ref_quantize_weight_nv.argtypes = [vp, i64, i64, i64, vp, vp, vp]
    L.sharq_ref_quantize_weight_nv.restype = ctypes.c_int
    L.sharq_ref_linear_nv.argtypes = [i64, i64, i32, i32, vp, vp, vp, vp, vp, f32, i64, vp, vp, f32, vp, i64]
    L.sharq_ref_linear_nv.restype = ctypes.c_int
    L.sharq_ref_e4m3_code.argtypes = [f32]
    L.sharq_ref_e4m3_code.restype = ctypes.c_uint8
    L.sharq_ref_set_threads.argtypes = [ctypes.c_int]
    L.sharq_ref_max_threads.restype = ctypes.c_int
    return L


if __name__ == "__main__":
    build()
