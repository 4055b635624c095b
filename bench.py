"""Benchmark of the SharQ sparse-dense FP4 linear layer on one MI355X.

Default workload (the headline): one step = the whole hot path over one batch
of synthetic input -- for each of the three Llama-3.1-8B linear shapes at
M = 2048 tokens (QKV and gate/up with the fused RMSNorm, down without), the
fused preparation kernel followed by the two-path FP4 GEMM (2:4 backbone +
dense residual, MXFP4, bf16 output).  Weights are quantized once before
timing, as in inference.

Printed: one JSON line with the step throughput (TFLOP/s of the method's
algorithmic work F_alg = 2 M N K (1 + n/m) -- the dense residual GEMM plus the
n/m-sparse backbone GEMM -- prep time included; the executed work F_exec =
4 M N K, which counts the backbone's pruned zeros that gfx950 multiplies
anyway, and the plain linear's F_lin = 2 M N K beside it), the roofline of the
dominant kernel (the two-path GEMM, against the dense MXFP4 MFMA peak), the
preparation kernel's HBM rate on its algorithmic bytes, and the CPU oracle
timed on a bounded sample.  Beside the published MFMA peak the roofline also
reports the sustained FP4 MFMA rate this device reaches right after the timed
steps (libsharq_probe.so: back-to-back MFMAs on every SIMD, with the shader
clock it ran at): under such load the part runs well below its rated clock.
Per-kernel times come from HIP events on the
launch stream around every launch of the timed steps (the warmup steps carry
the same events, so a profiler's per-kernel mean over the run covers the
same regime).

Other workloads (--workload), one JSON line each:
  llama-decode  the same three linears at M = 1, 16, 64, 256 (weight-stream bound)
  qwen-nvfp4    Qwen2.5-7B gate/up and down at M = 4096, NVFP4 with the dynamic
                per-tensor scale pre-pass
  llama-nvfp4-pairs  the Llama prefill linears in the paper's own setting:
                NVFP4 with the 4:8 in-pairs backbone
  moe           Qwen3-30B-A3B expert layers, 4096 tokens, top-8 of 128 experts,
                4:8 backbone, grouped GEMMs
  llama-fused   the default step with the producer-side fusions of the data
                flow: the residual add fused into the qkv and gate/up
                preparations and SiLU.mul into the down projection's, whose
                input is the gate/up GEMM's own output
  ablation      the path combinations (Sparse, plain FP4 RTN, Dense+Dense,
                Sparse+Sparse, SharQ) on the Llama prefill linears, MXFP4 2:4
                and NVFP4 4:8 in pairs, and SharQ with HiF4 2:4: time per step
                and the output error against the unquantized product, per mode
--calibrate-copy MiB runs a plain device copy of that size (the reference
kernel for scaling the profiler's HBM byte counters) and nothing else.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--workload NAME] [--no-cpu-baseline]

The default warmup is 200 steps (about 0.1 s of the default workload): over
the first ~50 steps after start-up the step time falls by ~12% as the part
ramps its clocks, and the timed steps measure the steady state after it.
"""

from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import platform
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))

METRIC = "SharQ linear TFLOPS (prep+2 FP4 GEMMs) & prep HBM GB/s, Llama-8B M=2048"
PEAK_FP4_TFLOPS = 10100.0     # MI355X dense MXFP4 MFMA
PEAK_16BIT_TFLOPS = 2500.0    # MI355X dense fp16 and bf16 MFMA
PEAK_HBM_GBPS = 8000.0        # MI355X HBM3E
T_TOKENS = 2048
N_INPUT_SETS = 2              # activations rotate between steps (defeats the 256 MB last-level cache)
DECODE_W_SETS = 5             # decode: weight copies rotate between steps (5 x 107 MB, past that cache)

# HBM traffic of the dominant kernel (k_linear_mx_persist<0>, the default workload with the dense backbone copy,
# mean over its three launch shapes), from two rocprofv3 --pmc runs
# (FETCH_SIZE x 2.0, WRITE_SIZE x 1.0: the factors a plain 1 GiB device copy
# gives).  Valid only for the GEMM source it was measured on (sha256 prefix);
# reported as null once that source has changed.
TRAFFIC = {"gemm_source": "54b1cdd92ca6fd6a", "bytes_per_launch": 270.32e6}
# the same for the MoE workload's k_linear_mx_grouped_persist<0> (mean of its gate_up and down launches)
MOE_TRAFFIC = {"gemm_source": "54b1cdd92ca6fd6a", "bytes_per_launch": 436.6e6}
# and for the Qwen2.5-7B NVFP4 workload's k_linear_nv_il (mean of its gate_up and down launches)
NV_TRAFFIC = {"gemm_source": "54b1cdd92ca6fd6a", "bytes_per_launch": 840.4e6}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gemm_flops(T, N, K):
    """Executed FP4 work of the two-path GEMM (F_exec): backbone (run dense,
    pruned zeros included) + residual."""
    return 4.0 * T * N * K


def alg_flops(T, N, K, n=2, m=4):
    """The method's algorithmic work (F_alg): the dense residual GEMM and the
    backbone GEMM over its n of every m positions."""
    return 2.0 * T * N * K * (1.0 + n / m)


def lin_flops(T, N, K):
    """The work of the plain linear layer Y = X W^T (F_lin)."""
    return 2.0 * T * N * K


def prep_bytes(T, K, norm, n=2, m=4, fmt="mx"):
    """Algorithmic HBM bytes of one preparation call: bf16 X (and gamma) in;
    backbone codes K n/m/2, metadata K/8, backbone scales K/32, residual codes
    K/2 and residual scales K/32 (MXFP4) or K/16 (NVFP4) out."""
    out = K * n / m / 2 + K / 8 + K / 32 + K / 2 + (K / 32 if fmt == "mx" else K / 16)
    return 2.0 * T * K + (2.0 * K if norm else 0.0) + T * out


def prep_bytes_written(T, K, norm, n=2, m=4, fmt="mx", backbone="compressed"):
    """Bytes a preparation call actually moves: as prep_bytes with the
    backbone stored compressed ("compressed"), as the dense copy beside it
    ("both", K/2 more per row) or as the dense copy alone ("dense-only": K/2
    instead of K n/m/2 + K/8)."""
    b = prep_bytes(T, K, norm, n, m, fmt)
    if backbone == "both":
        b += T * K / 2
    elif backbone == "dense-only":
        b += T * (K / 2 - K * n / m / 2 - K / 8)
    return b


def weight_bytes(N, K, fmt="mx"):
    """Bytes of the shared FP4 weight payload and the scales one GEMM reads."""
    return N * K / 2 + N * K / 32


def gemm_source_digest():
    with open(os.path.join(ROOT, "paper_2606_26587_amd", "csrc", "sharq_gemm.hip"), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def cpu_threads():
    try:
        from threadpoolctl import threadpool_info
        return int(max([p.get("num_threads", 1) for p in threadpool_info()] or [1]))
    except Exception:
        return 1


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return platform.processor() or None


def cpu_baseline(rows=768):
    """The CPU oracles on a bounded sample of the same step: `rows` of the 2048
    token rows of each Llama linear (preparation + two-path fp64 GEMM; the
    weights are quantized beforehand, untimed, as on the GPU).  The plain C
    oracle (oracle/sharq_ref.c, OpenMP over rows) is timed with one thread and
    with every host core for the preparation, and with every core for the
    GEMM; value is F_alg of the sample over its all-core time.  The NumPy
    oracle (element-wise preparation on one thread, BLAS float64 GEMM) is
    timed on the same sample beside it."""
    import ctypes as ct
    from oracle import build_ref
    from oracle import sharq_oracle as O
    from paper_2606_26587_amd import synth
    C = build_ref.load()
    cores = len(os.sched_getaffinity(0))

    def p(a):
        return ct.c_void_p(a.ctypes.data)

    flops = t_prep1 = t_prep = t_gemm = t_np_prep = t_np_gemm = 0.0
    for name, (K, N, norm) in synth.LLAMA_LINEARS.items():
        x = np.ascontiguousarray(synth.activations(T_TOKENS, K, seed=0)[:rows])
        g = synth.gamma(K, seed=0) if norm else None
        w = np.ascontiguousarray(synth.weight(N, K, seed=0))
        wc, ws = np.zeros((N, K // 2), np.uint8), np.zeros((N, K // 32), np.uint8)
        C.sharq_ref_set_threads(0)
        C.sharq_ref_quantize_weight(p(w), N, K, K, 0, p(wc), p(ws))
        bufs = [np.zeros((rows, K // 4), np.uint8), np.zeros((rows, K // 8), np.uint8),
                np.zeros((rows, K // 32), np.uint8), np.zeros((rows, K // 2), np.uint8),
                np.zeros((rows, K // 32), np.uint8)]
        args = [p(x), rows, K, K, None if g is None else p(g), ct.c_float(synth.LLAMA_EPS), 2, 4, 0,
                *(p(b) for b in bufs), None, None]
        for threads in (1, cores):
            C.sharq_ref_set_threads(threads)
            t0 = time.perf_counter()
            if C.sharq_ref_prepare(*args) != 0:
                raise RuntimeError("C oracle preparation failed")
            dt = time.perf_counter() - t0
            if threads == 1:
                t_prep1 += dt
            else:
                t_prep += dt
        Y = np.zeros((rows, N), np.float64)
        t0 = time.perf_counter()
        if C.sharq_ref_linear(rows, K, 2, 4, *(p(b) for b in bufs), N, p(wc), p(ws), p(Y), N) != 0:
            raise RuntimeError("C oracle GEMM failed")
        t_gemm += time.perf_counter() - t0
        # the NumPy oracle's GEMM reads the same weight bytes (the two oracles
        # quantize identically; their tests compare them byte for byte)
        wq = {"N": N, "K": K, "fmt": "mx", "codes": wc, "scale": ws, "scale_dn": ws, "tensor_scale": None}
        t0 = time.perf_counter()
        a = O.prepare(x, g, synth.LLAMA_EPS, 2, 4, "mx")
        t1 = time.perf_counter()
        O.linear(a, wq)
        t_np_prep += t1 - t0
        t_np_gemm += time.perf_counter() - t1
        flops += alg_flops(rows, N, K)
    C.sharq_ref_set_threads(0)
    return {"value": flops / (t_prep + t_gemm) / 1e12, "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"{rows} of the {T_TOKENS} token rows of each Llama linear (qkv, gate_up, down): the C "
                      f"oracle's preparation and fp64 two-path GEMM on all {cores} host cores; weight quantization "
                      f"untimed",
            "seconds": t_prep + t_gemm, "prep_seconds_1_thread": t_prep1, "prep_seconds_all_cores": t_prep,
            "gemm_seconds_all_cores": t_gemm, "prep_speedup_all_cores": t_prep1 / max(t_prep, 1e-12),
            "numpy_oracle": {"value": flops / (t_np_prep + t_np_gemm) / 1e12, "unit": "TFLOP/s",
                             "prep_seconds_1_thread": t_np_prep, "gemm_seconds_blas": t_np_gemm,
                             "blas_threads": cpu_threads()},
            "host_cpus": cores, "cpu": cpu_model()}


class HipEvent:
    """A timing-only HIP event created with hipEventDisableSystemFence: its
    record carries no system-scope release, so it does not write back and
    invalidate the caches between the kernels it brackets (with the default
    flags every record left a gap of ~6 us between kernels on MI355X).  The
    calls go to the HIP runtime torch has loaded (one libamdhip64.so.7 per
    process)."""

    DISABLE_SYSTEM_FENCE = 0x20000000
    _lib = None

    @classmethod
    def lib(cls):
        if cls._lib is None:
            L = ctypes.CDLL("libamdhip64.so.7")
            L.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            L.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            L.hipEventSynchronize.argtypes = [ctypes.c_void_p]
            L.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            L.hipEventDestroy.argtypes = [ctypes.c_void_p]
            cls._lib = L
        return cls._lib

    def __init__(self):
        self.h = ctypes.c_void_p()
        if self.lib().hipEventCreateWithFlags(ctypes.byref(self.h), self.DISABLE_SYSTEM_FENCE) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self, stream):
        if self.lib().hipEventRecord(self.h, ctypes.c_void_p(stream.cuda_stream)) != 0:
            raise RuntimeError("hipEventRecord failed")

    def elapsed_time(self, end) -> float:
        """Milliseconds from this event to `end` (both recorded)."""
        self.lib().hipEventSynchronize(end.h)
        ms = ctypes.c_float()
        if self.lib().hipEventElapsedTime(ctypes.byref(ms), self.h, end.h) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return float(ms.value)

    def __del__(self):
        if self._lib is not None and self.h:
            self._lib.hipEventDestroy(self.h)


class Timer:
    """Brackets every op of a step with HIP events on the launch stream."""

    def __init__(self, torch, stream, n_ops, steps):
        self.stream = stream
        self.ev = [[HipEvent() for _ in range(n_ops + 1)] for _ in range(steps)]

    def mark(self, step, i):
        self.ev[step][i].record(self.stream)

    def op_ms(self, i):
        return float(np.mean([e[i].elapsed_time(e[i + 1]) for e in self.ev]))


def tenths(values):
    """Means of `values` over (up to) ten consecutive, nearly equal parts."""
    if not values:
        return []
    return [float(np.mean(c)) for c in np.array_split(np.asarray(values, dtype=np.float64), min(10, len(values)))]


def run_steps(torch, stream, step, n_ops, steps, warmup):
    """Warm up, then time exactly `steps` steps synchronized on both sides.
    Every op of every step -- warmup and timed alike -- is bracketed by HIP
    events on the launch stream, so the per-kernel times are those of the
    timed steps themselves and a profiler's per-kernel mean over the whole run
    sees the same launch pattern."""
    tw = Timer(torch, stream, n_ops, max(warmup, 1))
    for i in range(warmup):
        step(i, lambda k, i=i: tw.mark(i, k))
    torch.cuda.synchronize()
    # step times over the warmup, in tenths: the part reaches its steady
    # clocks only after tens of milliseconds of load
    ramp = [tw.ev[i][0].elapsed_time(tw.ev[i][n_ops]) for i in range(warmup)]
    tm = Timer(torch, stream, n_ops, steps)
    t0, t1 = HipEvent(), HipEvent()
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record(stream)
    for i in range(steps):
        step(i, lambda k, i=i: tm.mark(i, k))
    t1.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    tm.warmup_ramp_ms = tenths(ramp)
    return t0.elapsed_time(t1) / steps, wall * 1e3 / steps, tm


def base_record(args, metric, value, unit, ms_step, dtype, config):
    return {"metric": metric, "value": value, "unit": unit, "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
            "vs_baseline": None, "dtype": dtype, "data": "synthetic", "config": config}


# ---------------------------------------------------------------------------
# workloads
# ---------------------------------------------------------------------------

def dense_layers(torch, S, synth, dev, shapes, T, fmt, n, m, n_sets, pairs=False, backbone="compressed", w_sets=1):
    def to_dev(u16):
        return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).to(dev)
    layers = []
    for name, (K, N, norm) in shapes.items():
        xs = [to_dev(synth.activations(T, K, seed=s)) for s in range(n_sets)]
        g = to_dev(synth.gamma(K, seed=0)) if norm else None
        wsrc = to_dev(synth.weight(N, K, seed=0))
        w = [S.sharq_quantize_weight(wsrc, fmt) for _ in range(w_sets)]   # copies at distinct addresses
        del wsrc
        acts = [S.alloc_act(T, K, n, m, fmt, dev, pairs, dense_backbone=backbone == "both",
                            dense_only=backbone == "dense-only") for _ in range(n_sets)]
        ys = [torch.empty((T, N), dtype=torch.bfloat16, device=dev) for _ in range(n_sets)]
        layers.append(dict(name=name, K=K, N=N, norm=norm, xs=xs, g=g, w=w, acts=acts, ys=ys))
    torch.cuda.synchronize()
    return layers


def dense_step(S, layers, stream, eps, n, m, fmt, n_sets, pairs=False):
    def step(i, mark):
        j = i % n_sets
        for li, L in enumerate(layers):
            if mark:
                mark(2 * li)
            S.sharq_prepare(L["xs"][j], L["g"], eps, n, m, fmt, out=L["acts"][j], stream=stream, pairs=pairs)
            if mark:
                mark(2 * li + 1)
            S.sharq_linear(L["acts"][j], L["w"][i % len(L["w"])], out=L["ys"][j], stream=stream)
        if mark:
            mark(2 * len(layers))
    return step


def per_linear(layers, tm, T, fmt, n, m, backbone="compressed"):
    per = []
    for li, L in enumerate(layers):
        prep_ms, gemm_ms = tm.op_ms(2 * li), tm.op_ms(2 * li + 1)
        f = alg_flops(T, L["N"], L["K"], n, m)
        fx = gemm_flops(T, L["N"], L["K"])
        b = prep_bytes(T, L["K"], L["norm"], n, m, fmt)
        bw = prep_bytes_written(T, L["K"], L["norm"], n, m, fmt, backbone)
        wb = weight_bytes(L["N"], L["K"], fmt)
        per.append({"linear": L["name"], "K": L["K"], "N": L["N"], "rmsnorm": L["norm"],
                    "prep_us": prep_ms * 1e3, "prep_bytes": b, "prep_GBps": b / (prep_ms * 1e-3) / 1e9,
                    "prep_bytes_moved": bw, "gemm_us": gemm_ms * 1e3, "gemm_flops_alg": f,
                    "gemm_TFLOPs": f / (gemm_ms * 1e-3) / 1e12, "gemm_flops_exec": fx,
                    "gemm_TFLOPs_exec": fx / (gemm_ms * 1e-3) / 1e12,
                    "weight_bytes": wb, "weight_GBps": wb / (gemm_ms * 1e-3) / 1e9})
        log(f"[bench] {L['name']:8s} T={T:5d} prep {prep_ms * 1e3:8.2f} us {per[-1]['prep_GBps']:8.1f} GB/s | "
            f"gemm {gemm_ms * 1e3:8.2f} us {per[-1]['gemm_TFLOPs']:8.1f} TFLOP/s alg "
            f"({per[-1]['gemm_TFLOPs_exec']:.1f} exec) {per[-1]['weight_GBps']:8.1f} GB/s of weight")
    return per


def copy_same_bytes(torch, dev, stream, nbytes, reps=20):
    """Mean time of a plain streaming device kernel moving `nbytes` (half
    read, half written), with sources rotated past the 256 MB last-level
    cache: the rate a copy reaches at this transfer size."""
    n = int(nbytes // 2) // 16 * 4   # int32 elements, 16-byte multiple
    nsrc = max(2, int((512 << 20) // max(4 * n, 1)) + 1)
    srcs = [torch.full((n,), i, dtype=torch.int32, device=dev) for i in range(nsrc)]
    dst = torch.empty(n, dtype=torch.int32, device=dev)
    with torch.cuda.stream(stream):
        # a streaming elementwise kernel (one read, one write per element);
        # torch's copy_ would go to the runtime's blit kernel instead
        for i in range(3):
            torch.bitwise_not(srcs[i % nsrc], out=dst)
        ev = [HipEvent() for _ in range(reps + 1)]
        ev[0].record(stream)
        for i in range(reps):
            torch.bitwise_not(srcs[i % nsrc], out=dst)
            ev[i + 1].record(stream)
    torch.cuda.synchronize()
    us = float(np.mean([ev[i].elapsed_time(ev[i + 1]) for i in range(reps)])) * 1e3
    del srcs, dst
    torch.cuda.empty_cache()
    return us


PROBE_ITERS = 2500               # ~1.7 ms of back-to-back MFMAs per probe launch


PROBES = {  # instruction: (entry point, flops per MFMA, description)
    "fp4": ("sharq_probe_mfma_fp4", 2.0 * 32 * 32 * 64,
            "back-to-back v_mfma_scale_f32_32x32x64_f8f6f4 (E2M1), 4 wavefronts x 8 accumulators per CU"),
    "bf16": ("sharq_probe_mfma_bf16", 2.0 * 32 * 32 * 16,
             "back-to-back v_mfma_f32_32x32x16_bf16, 4 wavefronts x 8 accumulators per CU"),
    "f16": ("sharq_probe_mfma_f16", 2.0 * 32 * 32 * 16,
            "back-to-back v_mfma_f32_32x32x16_f16, 4 wavefronts x 8 accumulators per CU"),
}


def mfma_probe(torch, dev, stream, iters=PROBE_ITERS, reps=3, kind="fp4"):
    """The sustained MFMA rate of this device for one instruction
    (libsharq_probe.so: four wavefronts per CU issuing independent 32x32 MFMAs
    -- the scaled FP4 one the MXFP4 GEMM runs on, the fp16 one of the NVFP4
    GEMM, or the bf16 one of the HiF4 GEMM), and the shader clock the probe ran at (shader-clock
    cycles over 100 MHz real-time ticks, averaged over the workgroups of the
    last launch).  This is the executed-work ceiling of a GEMM on that
    instruction on the part as it runs under that load, beside the published
    peak at the rated clock."""
    name, flops_per_mfma, desc = PROBES[kind]
    peak = PEAK_FP4_TFLOPS if kind == "fp4" else PEAK_16BIT_TFLOPS
    lib = ctypes.CDLL(os.path.join(ROOT, "paper_2606_26587_amd", "libsharq_probe.so"))
    fn = getattr(lib, name)
    fn.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
    fn.restype = ctypes.c_int
    cus = torch.cuda.get_device_properties(dev).multi_processor_count
    sink = torch.empty(cus * 256, dtype=torch.float32, device=dev)
    clk = torch.zeros(cus * 2, dtype=torch.int64, device=dev)
    ev = [HipEvent() for _ in range(reps + 2)]
    for i in range(reps + 1):   # launch 0 warms up
        ev[i].record(stream)
        rc = fn(iters, cus, sink.data_ptr(), clk.data_ptr(), stream.cuda_stream)
        if rc != 0:
            raise RuntimeError(f"{name} failed: {rc}")
    ev[reps + 1].record(stream)
    torch.cuda.synchronize()
    us = sorted(ev[i].elapsed_time(ev[i + 1]) * 1e3 for i in range(1, reps + 1))
    c = clk.view(cus, 2).cpu().numpy().astype(np.float64)
    flops = cus * 4 * iters * 32 * flops_per_mfma
    med = us[len(us) // 2]
    return {"kernel": f"{name}: {desc}",
            "achieved": flops / (med * 1e-6) / 1e12, "unit": "TFLOP/s",
            "frac_of_peak": flops / (med * 1e-6) / 1e12 / peak,
            "clock_GHz": float(c[:, 0].sum() / c[:, 1].sum() * 0.1), "launch_us": us,
            "flops_per_launch": flops}


def nv_roofline(torch, dev, stream, per, t_gemm, measured=None):
    """The NVFP4 GEMMs' roofline record: algorithmic and executed work against
    the published 16-bit peak and against the sustained fp16 MFMA rate (the
    instruction the NVFP4 GEMM runs on for these K) measured right after the
    timed steps.  measured: the workload's HBM traffic record (NV_TRAFFIC), or None."""
    flops = sum(p["gemm_flops_alg"] for p in per)
    f_exec = sum(p["gemm_flops_exec"] for p in per)
    sus = mfma_probe(torch, dev, stream, kind="f16")
    log(f"[bench] fp16 MFMA probe: {sus['achieved']:.0f} TFLOP/s sustained at {sus['clock_GHz']:.2f} GHz; "
        f"GEMM executed work at {f_exec / t_gemm / 1e12 / sus['achieved']:.2f} of it")
    return {"bound": "mfma", "kernel": "k_linear_nv_il (fp16 MFMA over dequantized FP4)",
            "achieved": flops / t_gemm / 1e12, "peak": PEAK_16BIT_TFLOPS, "unit": "TFLOP/s",
            "frac": flops / t_gemm / 1e12 / PEAK_16BIT_TFLOPS, "flops": "F_alg",
            "traffic": (measured["bytes_per_launch"] if measured is not None
                        and measured["gemm_source"] == gemm_source_digest() else None),
            "achieved_exec": f_exec / t_gemm / 1e12, "frac_exec": f_exec / t_gemm / 1e12 / PEAK_16BIT_TFLOPS,
            "sustained_mfma": sus, "frac_exec_of_sustained": f_exec / t_gemm / 1e12 / sus["achieved"],
            "frac_alg_of_sustained": flops / t_gemm / 1e12 / sus["achieved"]}


def llama_prefill(args, torch, S, synth, dev, stream):
    backbone = args.backbone
    layers = dense_layers(torch, S, synth, dev, synth.LLAMA_LINEARS, T_TOKENS, "mx", 2, 4, N_INPUT_SETS,
                          backbone=backbone)
    log(f"[bench] set up {len(layers)} linears, M={T_TOKENS}, backbone stored {backbone}")
    step = dense_step(S, layers, stream, synth.LLAMA_EPS, 2, 4, "mx", N_INPUT_SETS)
    ms_step, wall_ms, tm = run_steps(torch, stream, step, 2 * len(layers), args.steps, args.warmup)
    log(f"[bench] timed {args.steps} steps: {ms_step:.4f} ms/step (wall {wall_ms:.4f} ms/step)")
    per = per_linear(layers, tm, T_TOKENS, "mx", 2, 4, backbone)
    f_alg = sum(p["gemm_flops_alg"] for p in per)
    f_exec = sum(p["gemm_flops_exec"] for p in per)
    f_lin = sum(lin_flops(T_TOKENS, p["N"], p["K"]) for p in per)
    t_gemm = sum(p["gemm_us"] for p in per) * 1e-6
    t_prep = sum(p["prep_us"] for p in per) * 1e-6
    bytes_prep = sum(p["prep_bytes"] for p in per)
    bytes_moved = sum(p["prep_bytes_moved"] for p in per)
    gemm_tf = f_alg / t_gemm / 1e12
    prep_gbps = bytes_prep / t_prep / 1e9
    traffic = None
    if TRAFFIC is not None and TRAFFIC["gemm_source"] == gemm_source_digest():
        traffic = TRAFFIC["bytes_per_launch"]
    step_s = ms_step * 1e-3
    out = base_record(
        args, METRIC, f_alg / step_s / 1e12, "TFLOP/s", ms_step, "mxfp4",
        {"workload": "Llama-3.1-8B prefill linears qkv (K4096,N6144,RMSNorm), gate_up (K4096,N28672,"
                     "RMSNorm), down (K14336,N4096); M=2048 tokens; 2:4 backbone; MXFP4; bf16 out",
         "tokens": T_TOKENS, "pattern": "2:4", "format": "MXFP4", "flops_per_step": f_alg,
         "backbone_for_gemm": {"dense-only": "dense copy alone, written by the preparation",
                               "both": "dense copy written beside the compressed backbone",
                               "compressed": "compressed, expanded in the GEMM"}[backbone],
         "flops_counting": "F_alg = 2*M*N*K*(1+n/m) per linear (dense residual GEMM + 2:4 backbone GEMM)",
         "flops_exec_per_step": f_exec, "flops_lin_per_step": f_lin,
         "exec_TFLOPs": f_exec / step_s / 1e12, "lin_TFLOPs": f_lin / step_s / 1e12})
    kern = {"dense-only": "k_linear_mx_persist<0> (two-path FP4 GEMM reading the dense backbone copy)",
            "both": "k_linear_mx_persist<0> (two-path FP4 GEMM reading the dense backbone copy)",
            "compressed": "k_linear_mx_persist<24> (two-path FP4 GEMM, backbone expanded in registers)"}[backbone]
    out["roofline"] = {"bound": "mfma", "kernel": kern, "achieved": gemm_tf,
                       "peak": PEAK_FP4_TFLOPS, "unit": "TFLOP/s", "frac": gemm_tf / PEAK_FP4_TFLOPS,
                       "traffic": traffic, "flops_per_launch": f_alg / len(per),
                       "us_per_launch": t_gemm * 1e6 / len(per), "flops": "F_alg",
                       "achieved_exec": f_exec / t_gemm / 1e12, "frac_exec": f_exec / t_gemm / 1e12 / PEAK_FP4_TFLOPS,
                       "achieved_lin": f_lin / t_gemm / 1e12}
    out["prep"] = {"bound": "hbm", "kernel": "k_prep_norm_split (qkv, gate_up) / k_prep_blocks (down)",
                   "achieved": prep_gbps, "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": prep_gbps / PEAK_HBM_GBPS,
                   "bytes_per_step": bytes_prep,
                   "bytes": "2 M K (X) + 2 K (gamma) + M K (n/m/2 + 1/8 + 1/32 + 1/2 + 1/32) (prepared outputs)",
                   "bytes_moved_per_step": bytes_moved,
                   "moved_GBps": bytes_moved / t_prep / 1e9}
    # the same bytes moved by a plain device copy, one launch per linear
    copy_us = [copy_same_bytes(torch, dev, stream, p["prep_bytes"]) for p in per]
    for p, cu in zip(per, copy_us):
        p["copy_same_bytes_us"] = cu
    copy_gbps = bytes_prep / (sum(copy_us) * 1e-6) / 1e9
    out["prep"]["copy_same_bytes"] = {"achieved": copy_gbps, "unit": "GB/s", "frac": copy_gbps / PEAK_HBM_GBPS,
                                      "prep_vs_copy": prep_gbps / copy_gbps}
    # the sustained FP4 MFMA rate of this device, measured after the timed steps
    sus = mfma_probe(torch, dev, stream)
    out["roofline"]["sustained_mfma"] = sus
    out["roofline"]["frac_exec_of_sustained"] = f_exec / t_gemm / 1e12 / sus["achieved"]
    out["roofline"]["frac_alg_of_sustained"] = gemm_tf / sus["achieved"]
    log(f"[bench] FP4 MFMA probe: {sus['achieved']:.0f} TFLOP/s sustained at {sus['clock_GHz']:.2f} GHz; "
        f"GEMM executed work at {f_exec / t_gemm / 1e12 / sus['achieved']:.2f} of it")
    log(f"[bench] prep {prep_gbps:.0f} GB/s algorithmic ({bytes_moved / t_prep / 1e9:.0f} GB/s moved); "
        f"a device copy of the same bytes {copy_gbps:.0f} GB/s; GEMM {gemm_tf:.0f} TFLOP/s alg, "
        f"{f_exec / t_gemm / 1e12:.0f} exec")
    out["per_linear"] = per
    out["wall_ms_per_step"] = wall_ms
    out["warmup_ramp_ms"] = tm.warmup_ramp_ms
    log("[bench] step time over the warmup, by tenths (ms): " + " ".join(f"{v:.3f}" for v in tm.warmup_ramp_ms))
    return out


def llama_decode(args, torch, S, synth, dev, stream):
    """Decode: the three Llama linears at M = 1 ... 256 tokens, weight copies
    rotated past the last-level cache.  Each M is timed twice: the
    preparation and the GEMM as two launches, and through
    sharq_prepare_linear, which runs both in one kernel for a few rows."""
    outs = []
    for T in (1, 2, 4, 16, 64, 256):
        layers = dense_layers(torch, S, synth, dev, synth.LLAMA_LINEARS, T, "mx", 2, 4, 1, w_sets=DECODE_W_SETS)
        step = dense_step(S, layers, stream, synth.LLAMA_EPS, 2, 4, "mx", 1)
        ms_step, wall_ms, tm = run_steps(torch, stream, step, 2 * len(layers), args.steps, args.warmup)
        per = per_linear(layers, tm, T, "mx", 2, 4)

        def fused_step(i, mark):
            for li, L in enumerate(layers):
                if mark:
                    mark(li)
                S.sharq_prepare_linear(L["xs"][0], L["g"], L["w"][i % len(L["w"])], synth.LLAMA_EPS, 2, 4, "mx",
                                       act=L["acts"][0], out=L["ys"][0], stream=stream)
            if mark:
                mark(len(layers))

        ms_fused, _, tf = run_steps(torch, stream, fused_step, len(layers), args.steps, args.warmup)
        for li, p in enumerate(per):
            p["prepare_linear_us"] = tf.op_ms(li) * 1e3
            p["separate_us"] = p["prep_us"] + p["gemm_us"]
        wb = sum(p["weight_bytes"] for p in per)
        t_gemm = sum(p["gemm_us"] for p in per) * 1e-6
        log(f"[bench] decode M={T}: separate {ms_step * 1e3:.1f} us/step, one call {ms_fused * 1e3:.1f} us/step; "
            + ", ".join(f"{p['linear']} {p['separate_us']:.1f} -> {p['prepare_linear_us']:.1f}" for p in per))
        out = base_record(args, "SharQ decode linears weight-stream GB/s (prep+GEMM), Llama-8B",
                          wb / (ms_step * 1e-3) / 1e9, "GB/s", ms_step, "mxfp4",
                          {"workload": f"Llama-3.1-8B decode linears qkv, gate_up, down; M={T}; 2:4; MXFP4",
                           "tokens": T})
        out["roofline"] = {"bound": "hbm", "kernel": "k_linear_mx_skinny / k_linear_mx_persist",
                           "achieved": wb / t_gemm / 1e9, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                           "frac": wb / t_gemm / 1e9 / PEAK_HBM_GBPS, "traffic": None}
        out["prepare_linear_ms_per_step"] = ms_fused
        out["per_linear"] = per
        outs.append(out)
        del layers
        torch.cuda.empty_cache()
    return outs


def qwen_nvfp4(args, torch, S, synth, dev, stream):
    T = 4096
    layers = dense_layers(torch, S, synth, dev, synth.QWEN_LINEARS, T, "nv", 2, 4, N_INPUT_SETS,
                          backbone=args.backbone)
    step = dense_step(S, layers, stream, 1e-6, 2, 4, "nv", N_INPUT_SETS)
    ms_step, wall_ms, tm = run_steps(torch, stream, step, 2 * len(layers), args.steps, args.warmup)
    per = per_linear(layers, tm, T, "nv", 2, 4, args.backbone)
    flops = sum(p["gemm_flops_alg"] for p in per)
    t_gemm = sum(p["gemm_us"] for p in per) * 1e-6
    t_prep = sum(p["prep_us"] for p in per) * 1e-6
    pb = sum(p["prep_bytes"] for p in per)
    out = base_record(args, "SharQ linear TFLOPS (prep+2 FP4 GEMMs), Qwen2.5-7B M=4096 NVFP4",
                      flops / (ms_step * 1e-3) / 1e12, "TFLOP/s", ms_step, "nvfp4",
                      {"workload": "Qwen2.5-7B prefill linears gate_up (K3584,N37888,RMSNorm), down (K18944,N3584); "
                                   "M=4096; 2:4; NVFP4 with dynamic per-tensor scale", "tokens": T,
                       "backbone_for_gemm": args.backbone})
    out["roofline"] = nv_roofline(torch, dev, stream, per, t_gemm,
                                  NV_TRAFFIC if args.backbone == "dense-only" else None)
    out["prep"] = {"bound": "hbm", "achieved": pb / t_prep / 1e9, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                   "frac": pb / t_prep / 1e9 / PEAK_HBM_GBPS,
                   "note": "time includes the per-tensor amax pre-pass (a second read of X)"}
    out["per_linear"] = per
    return out


def llama_nvfp4_pairs(args, torch, S, synth, dev, stream):
    """The paper's own instantiation on the headline shapes: NVFP4 with the
    4:8 in-pairs backbone, Llama-3.1-8B prefill linears at M = 2048."""
    layers = dense_layers(torch, S, synth, dev, synth.LLAMA_LINEARS, T_TOKENS, "nv", 4, 8, N_INPUT_SETS, True,
                          backbone=args.backbone)
    step = dense_step(S, layers, stream, synth.LLAMA_EPS, 4, 8, "nv", N_INPUT_SETS, True)
    ms_step, wall_ms, tm = run_steps(torch, stream, step, 2 * len(layers), args.steps, args.warmup)
    per = per_linear(layers, tm, T_TOKENS, "nv", 4, 8, args.backbone)
    flops = sum(p["gemm_flops_alg"] for p in per)
    t_gemm = sum(p["gemm_us"] for p in per) * 1e-6
    t_prep = sum(p["prep_us"] for p in per) * 1e-6
    pb = sum(p["prep_bytes"] for p in per)
    out = base_record(args, "SharQ linear TFLOPS (prep+2 FP4 GEMMs), Llama-8B M=2048, NVFP4 4:8 in pairs",
                      flops / (ms_step * 1e-3) / 1e12, "TFLOP/s", ms_step, "nvfp4",
                      {"workload": "Llama-3.1-8B prefill linears qkv, gate_up (RMSNorm), down; M=2048; "
                                   "4:8 in pairs; NVFP4 with dynamic per-tensor scale", "tokens": T_TOKENS,
                       "backbone_for_gemm": args.backbone})
    out["roofline"] = nv_roofline(torch, dev, stream, per, t_gemm)
    out["prep"] = {"bound": "hbm", "achieved": pb / t_prep / 1e9, "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                   "frac": pb / t_prep / 1e9 / PEAK_HBM_GBPS,
                   "note": "time includes the per-tensor amax pre-pass (a second read of X)"}
    out["per_linear"] = per
    return out


def moe(args, torch, S, synth, dev, stream):
    cfg = synth.MOE
    T, H, E, I, k = cfg["tokens"], cfg["hidden"], cfg["experts"], cfg["inter"], cfg["topk"]

    def to_dev(u16):
        return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).to(dev)

    x = to_dev(synth.activations(T, H, seed=0))
    g = to_dev(synth.gamma(H, seed=0))
    ridx, offs = synth.router_topk(T, E, k, seed=0)
    total = int(offs[-1])
    h = to_dev(synth.activations(total, I, seed=1))   # stands in for SiLU(gate) * up, expert-sorted
    log(f"[bench] moe: quantizing {E} experts x (gate_up {2 * I}x{H}, down {H}x{I})")
    w_gu = S.stack_weights([S.sharq_quantize_weight(to_dev(synth.weight(2 * I, H, seed=100 + e)), "mx")
                            for e in range(E)])
    w_dn = S.stack_weights([S.sharq_quantize_weight(to_dev(synth.weight(H, I, seed=1000 + e)), "mx")
                            for e in range(E)])
    ri = torch.from_numpy(ridx).to(dev)
    of = torch.from_numpy(offs).to(dev)
    a1 = S.alloc_act(T, H, 4, 8, "mx", dev, dense_only=True)
    a2 = S.alloc_act(total, I, 4, 8, "mx", dev, dense_only=True)
    y1 = torch.empty((total, 2 * I), dtype=torch.bfloat16, device=dev)
    y2 = torch.empty((total, H), dtype=torch.bfloat16, device=dev)
    torch.cuda.synchronize()

    def step(i, mark):
        if mark:
            mark(0)
        S.sharq_prepare(x, g, 1e-6, 4, 8, "mx", out=a1, stream=stream)
        if mark:
            mark(1)
        S.sharq_linear_grouped(a1, ri, of, total, w_gu, out=y1, stream=stream)
        if mark:
            mark(2)
        S.sharq_prepare(h, None, 1e-6, 4, 8, "mx", out=a2, stream=stream)
        if mark:
            mark(3)
        S.sharq_linear_grouped(a2, None, of, total, w_dn, out=y2, stream=stream)
        if mark:
            mark(4)

    ms_step, wall_ms, tm = run_steps(torch, stream, step, 4, args.steps, args.warmup)
    f1, f2 = alg_flops(total, 2 * I, H, 4, 8), alg_flops(total, H, I, 4, 8)
    ops = {"prep_gate_up_us": tm.op_ms(0) * 1e3, "grouped_gate_up_us": tm.op_ms(1) * 1e3,
           "prep_down_us": tm.op_ms(2) * 1e3, "grouped_down_us": tm.op_ms(3) * 1e3}
    t_g = (tm.op_ms(1) + tm.op_ms(3)) * 1e-3
    log(f"[bench] moe {ops}")
    out = base_record(args, "SharQ MoE expert layers TFLOPS (prep+grouped FP4 GEMMs), Qwen3-30B-A3B 4096 tokens",
                      (f1 + f2) / (ms_step * 1e-3) / 1e12, "TFLOP/s", ms_step, "mxfp4",
                      {"workload": f"Qwen3-30B-A3B experts: {T} tokens, top-{k} of {E}, gate_up {2 * I}x{H} "
                                   f"(RMSNorm), down {H}x{I}; 4:8; MXFP4", "tokens": T, "routed_rows": total})
    traffic = None
    if MOE_TRAFFIC is not None and MOE_TRAFFIC["gemm_source"] == gemm_source_digest():
        traffic = MOE_TRAFFIC["bytes_per_launch"]
    out["roofline"] = {"bound": "mfma",
                       "kernel": "k_linear_mx_grouped_persist<0> (grouped two-path FP4 GEMM reading the dense "
                                 "backbone copy)",
                       "achieved": (f1 + f2) / t_g / 1e12, "peak": PEAK_FP4_TFLOPS, "unit": "TFLOP/s",
                       "frac": (f1 + f2) / t_g / 1e12 / PEAK_FP4_TFLOPS, "traffic": traffic, "flops": "F_alg",
                       "traffic_note": "HBM-side bytes per launch (FETCH_SIZE + WRITE_SIZE, scaled by a plain "
                                       "copy's counters), mean of the gate_up and down launches"}
    out["ops"] = ops
    return out


def llama_fused(args, torch, S, synth, dev, stream):
    """The Llama-3.1-8B prefill linears at M = 2048 with the producer-side
    fusions of a transformer block's data flow: h = bf16(x + res) fused into
    the RMSNorm preparation of qkv and of gate/up (h written back to the
    residual stream in place), and h = bf16(SiLU(gate) * up) fused into the
    down projection's preparation, read from the gate/up GEMM's output."""
    def to_dev(u16):
        return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).to(dev)

    T, eps = T_TOKENS, synth.LLAMA_EPS
    L = {}
    for name, (K, N, norm) in synth.LLAMA_LINEARS.items():
        L[name] = dict(K=K, N=N, norm=norm, w=S.sharq_quantize_weight(to_dev(synth.weight(N, K, seed=0))),
                       g=to_dev(synth.gamma(K, seed=0)) if norm else None,
                       act=S.alloc_act(T, K, 2, 4, "mx", dev, dense_only=True),
                       y=torch.empty((T, N), dtype=torch.bfloat16, device=dev))
    H = synth.LLAMA_LINEARS["qkv"][0]
    I = synth.LLAMA_LINEARS["down"][0]
    x_in = [to_dev(synth.activations(T, H, seed=s)) for s in range(N_INPUT_SETS)]
    attn = [to_dev(synth.activations(T, H, seed=10 + s)) for s in range(N_INPUT_SETS)]
    res0 = to_dev(synth.activations(T, H, seed=20))
    res = res0.clone()
    torch.cuda.synchronize()

    def step(i, mark):
        j = i % N_INPUT_SETS
        q, gu, dn = L["qkv"], L["gate_up"], L["down"]
        if mark:
            mark(0)
        S.sharq_prepare_residual(x_in[j], res, q["g"], eps, 2, 4, "mx", h_out=res, out=q["act"], stream=stream)
        if mark:
            mark(1)
        S.sharq_linear(q["act"], q["w"], out=q["y"], stream=stream)
        if mark:
            mark(2)
        S.sharq_prepare_residual(attn[j], res, gu["g"], eps, 2, 4, "mx", h_out=res, out=gu["act"], stream=stream)
        if mark:
            mark(3)
        S.sharq_linear(gu["act"], gu["w"], out=gu["y"], stream=stream)
        if mark:
            mark(4)
        S.sharq_prepare_silu_mul(gu["y"][:, :I], gu["y"][:, I:], 2, 4, "mx", out=dn["act"], stream=stream)
        if mark:
            mark(5)
        S.sharq_linear(dn["act"], dn["w"], out=dn["y"], stream=stream)
        if mark:
            mark(6)

    ms_step, wall_ms, tm = run_steps(torch, stream, step, 6, args.steps, args.warmup)
    flops = sum(alg_flops(T, v["N"], v["K"]) for v in L.values())
    # algorithmic bytes of the fused preparations: x and res read, h written
    # (and gamma read) for the residual adds; gate and up read for SiLU.mul;
    # the prepared activation written (0.9375 B per element at MXFP4 2:4)
    b_res = 3 * 2.0 * T * H + 2.0 * H + 0.9375 * T * H
    b_silu = 2 * 2.0 * T * I + 0.9375 * T * I
    ops = {"prep_residual_qkv_us": tm.op_ms(0) * 1e3, "gemm_qkv_us": tm.op_ms(1) * 1e3,
           "prep_residual_gate_up_us": tm.op_ms(2) * 1e3, "gemm_gate_up_us": tm.op_ms(3) * 1e3,
           "prep_silu_mul_down_us": tm.op_ms(4) * 1e3, "gemm_down_us": tm.op_ms(5) * 1e3}
    ops["prep_residual_GBps"] = b_res / (tm.op_ms(0) * 1e-3) / 1e9
    ops["prep_silu_mul_GBps"] = b_silu / (tm.op_ms(4) * 1e-3) / 1e9
    log(f"[bench] fused data flow {ms_step:.4f} ms/step: " + ", ".join(f"{k} {v:.1f}" for k, v in ops.items()))
    out = base_record(args, "SharQ linear TFLOPS (fused prep+2 FP4 GEMMs), Llama-8B M=2048, fused data flow",
                      flops / (ms_step * 1e-3) / 1e12, "TFLOP/s", ms_step, "mxfp4",
                      {"workload": "Llama-3.1-8B prefill linears with the residual add fused into the qkv and "
                                   "gate_up preparations and SiLU.mul fused into the down preparation (input = the "
                                   "gate_up output); M=2048; 2:4; MXFP4; bf16 out", "tokens": T})
    out["ops"] = ops
    return out


ABLATION_MODES = ["sharq", "sparse", "dense", "dense_dense", "sparse_sparse"]
MODE_PATHS = {"sharq": 2, "sparse": 1, "dense": 1, "dense_dense": 2, "sparse_sparse": 2}


def ablation(args, torch, S, synth, dev, stream):
    """Path combinations (the paper's ablation over sparse / dense paths) on
    the Llama-3.1-8B prefill linears at M = 2048, in MXFP4 2:4 and in the
    paper's NVFP4 4:8-in-pairs setting.  Per mode: the step time (prep + GEMM
    of the three linears) and, as an accuracy proxy that needs no dataset, the
    mean per-row relative error of Y against the unquantized product y W^T
    (fp32; weight quantization included, the same for every mode)."""
    def to_dev(u16):
        return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).to(dev)

    T = T_TOKENS
    eps = synth.LLAMA_EPS
    outs = []
    for fmt, n, m, pairs in (("mx", 2, 4, False), ("nv", 4, 8, True), ("hif4", 2, 4, False)):
        layers = []
        for name, (K, N, norm) in synth.LLAMA_LINEARS.items():
            x = to_dev(synth.activations(T, K, seed=0))
            g = to_dev(synth.gamma(K, seed=0)) if norm else None
            w_bf = to_dev(synth.weight(N, K, seed=0))
            # the unquantized product, in fp32: y = RMSNorm(x) * gamma (or x), Y = y W^T
            xf = x.float()
            if norm:
                r = torch.rsqrt(xf.pow(2).mean(dim=1, keepdim=True) + eps)
                yf = (xf * r) * g.float()[None, :]
            else:
                yf = xf
            yref = yf @ w_bf.float().t().contiguous()
            layers.append(dict(name=name, K=K, N=N, norm=norm, x=x, g=g, w=S.sharq_quantize_weight(w_bf, fmt),
                               yref=yref, y=torch.empty((T, N), dtype=torch.float32, device=dev)))
            del xf, yf
        torch.cuda.synchronize()
        res = {}
        # HiF4 is built for the method's own combination only
        for mode in (ABLATION_MODES if fmt != "hif4" else ["sharq"]):
            # SharQ stores its backbone as the benchmark's --backbone says (HiF4: compressed)
            bb = args.backbone if mode == "sharq" and fmt != "hif4" else "compressed"
            acts = [S.alloc_act(T, L["K"], n, m, fmt, dev, pairs, mode, dense_backbone=bb == "both",
                                dense_only=bb == "dense-only") for L in layers]

            def step(i, mark, acts=acts):
                for li, L in enumerate(layers):
                    if mark:
                        mark(2 * li)
                    S.sharq_prepare(L["x"], L["g"], eps, n, m, fmt, out=acts[li], stream=stream, pairs=pairs)
                    if mark:
                        mark(2 * li + 1)
                    S.sharq_linear(acts[li], L["w"], out=L["y"], stream=stream)
                if mark:
                    mark(2 * len(layers))

            ms_step, _, tm = run_steps(torch, stream, step, 2 * len(layers), args.steps, args.warmup)
            errs = {}
            for L in layers:
                d = (L["y"] - L["yref"]).norm(dim=1) / L["yref"].norm(dim=1).clamp_min(1e-30)
                errs[L["name"]] = float(d.mean())
            flops = sum(2.0 * MODE_PATHS[mode] * T * L["N"] * L["K"] for L in layers)
            res[mode] = {"ms_per_step": ms_step, "executed_TFLOPs": flops / (ms_step * 1e-3) / 1e12,
                         "prep_us": [tm.op_ms(2 * li) * 1e3 for li in range(len(layers))],
                         "gemm_us": [tm.op_ms(2 * li + 1) * 1e3 for li in range(len(layers))],
                         "rel_err": errs, "rel_err_mean": float(np.mean(list(errs.values())))}
            log(f"[bench] ablation {fmt} {mode:14s} {ms_step:7.4f} ms/step  rel err "
                + "  ".join(f"{k} {v:.4f}" for k, v in errs.items()))
            del acts
        setting = {"mx": "MXFP4 2:4", "nv": "NVFP4 4:8 in pairs", "hif4": "HiF4 2:4"}[fmt]
        out = base_record(args, "SharQ path-combination ablation: time per step and output error, Llama-8B M=2048",
                          res["sharq"]["executed_TFLOPs"], "TFLOP/s", res["sharq"]["ms_per_step"],
                          {"mx": "mxfp4", "nv": "nvfp4", "hif4": "hif4"}[fmt],
                          {"workload": f"Llama-3.1-8B prefill linears qkv, gate_up (RMSNorm), down; M=2048; "
                                       f"{setting}; fp32 out; modes " + ", ".join(res), "tokens": T,
                           "sharq_backbone": args.backbone if fmt != "hif4" else "compressed"})
        out["modes"] = res
        out["error_definition"] = ("mean over token rows of |Y_t - y_t W^T| / |y_t W^T| (fp32 reference with the "
                                   "unquantized weight), per linear")
        outs.append(out)
        del layers
        torch.cuda.empty_cache()
    return outs


def calibrate_copy(torch, dev, mib):
    n = mib * (1 << 20)
    src = torch.empty(n, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty_like(src)
    for _ in range(5):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"calibrate_copy_bytes": n, "launches": 5}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=200,
                    help="untimed steps first: the part needs tens of milliseconds of load to reach its steady "
                         "clocks (the step time over the warmup is reported by tenths)")
    ap.add_argument("--workload", default="llama-prefill",
                    choices=["llama-prefill", "llama-decode", "qwen-nvfp4", "llama-nvfp4-pairs", "moe",
                             "ablation", "llama-fused"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--backbone", default="dense-only", choices=["dense-only", "both", "compressed"],
                    help="prefill and the NVFP4 workloads: how the preparation stores the backbone for the "
                         "GEMM -- the dense copy alone (default), the dense copy beside the compressed form, or "
                         "the compressed form only (the GEMM then expands it)")
    ap.add_argument("--cpu-rows", type=int, default=768)
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MiB")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the layer shards by token rows or weight columns without kernel changes)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_26587_amd import sharq as S
    from paper_2606_26587_amd import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()
    if args.calibrate_copy:
        calibrate_copy(torch, dev, args.calibrate_copy)
        return

    if args.workload == "llama-prefill":
        out = llama_prefill(args, torch, S, synth, dev, stream)
        if not args.no_cpu_baseline:
            log("[bench] timing the CPU oracle on a bounded sample ...")
            out["cpu_baseline"] = cpu_baseline(args.cpu_rows)
            log(f"[bench] cpu oracle: {out['cpu_baseline']['value']:.4f} TFLOP/s "
                f"in {out['cpu_baseline']['seconds']:.1f} s")
        print(json.dumps(out), flush=True)
    elif args.workload == "llama-decode":
        for o in llama_decode(args, torch, S, synth, dev, stream):
            print(json.dumps(o), flush=True)
    elif args.workload == "qwen-nvfp4":
        print(json.dumps(qwen_nvfp4(args, torch, S, synth, dev, stream)), flush=True)
    elif args.workload == "llama-nvfp4-pairs":
        print(json.dumps(llama_nvfp4_pairs(args, torch, S, synth, dev, stream)), flush=True)
    elif args.workload == "llama-fused":
        print(json.dumps(llama_fused(args, torch, S, synth, dev, stream)), flush=True)
    elif args.workload == "ablation":
        for o in ablation(args, torch, S, synth, dev, stream):
            print(json.dumps(o), flush=True)
    else:
        print(json.dumps(moe(args, torch, S, synth, dev, stream)), flush=True)


if __name__ == "__main__":
    main()
