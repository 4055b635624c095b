"""Benchmark of the SharQ sparse-dense FP4 linear layer on one MI355X.

One step = the whole hot path over one batch of synthetic input: for each of
the three Llama-3.1-8B linear shapes at M = 2048 tokens (QKV and gate/up with
the fused RMSNorm, down without), the fused preparation kernel followed by the
two-path FP4 GEMM (2:4 backbone + dense residual, MXFP4, bf16 output).  Weights
are quantized once before timing, as in inference.

Printed: one JSON line with the step throughput (TFLOP/s over the two FP4
GEMMs' executed work, prep time included), the roofline of the dominant kernel
(the two-path GEMM, against the dense MXFP4 MFMA peak), the preparation
kernel's HBM rate, and the CPU oracle timed on a bounded sample.

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
"""

from __future__ import annotations

import argparse
import json
import os
import platform
import sys
import time

import numpy as np

METRIC = "SharQ linear TFLOPS (prep+2 FP4 GEMMs) & prep HBM GB/s, Llama-8B M=2048"
PEAK_FP4_TFLOPS = 10100.0     # MI355X dense MXFP4 MFMA
PEAK_HBM_GBPS = 8000.0        # MI355X HBM3E
T_TOKENS = 2048
N_INPUT_SETS = 2              # activations rotate between steps (defeats the 256 MB last-level cache)


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def gemm_flops(T, N, K):
    """Executed FP4 work of the two-path GEMM: backbone (expanded to dense) + residual."""
    return 4.0 * T * N * K


def prep_bytes(T, K, norm):
    """Algorithmic HBM bytes of one preparation call (MXFP4, 2:4): bf16 X and gamma in;
    backbone codes K/4, metadata K/8, two scale rows K/32 each, residual codes K/2 out."""
    return 2.0 * T * K + (2.0 * K if norm else 0.0) + T * (K / 4 + K / 8 + K / 32 + K / 2 + K / 32)


def cpu_baseline(rows=128):
    """The CPU oracle on a bounded sample of the same step: `rows` of the 2048
    token rows of each linear (preparation + two-path fp64 GEMM)."""
    from oracle import sharq_oracle as O
    from paper_2606_26587_amd import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threads = 1
    flops = 0.0
    elapsed = 0.0
    for name, (K, N, norm) in synth.LLAMA_LINEARS.items():
        x = synth.activations(T_TOKENS, K, seed=0)[:rows]
        g = synth.gamma(K, seed=0) if norm else None
        wq = O.quantize_weight(synth.weight(N, K, seed=0))
        t0 = time.perf_counter()
        a = O.prepare(x, g, synth.LLAMA_EPS, 2, 4, "mx")
        O.linear(a, wq)
        elapsed += time.perf_counter() - t0
        flops += gemm_flops(rows, N, K)
    return {"value": flops / elapsed / 1e12, "unit": "TFLOP/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{rows} of {T_TOKENS} token rows of each Llama linear (qkv, gate_up, down): "
                      f"NumPy preparation + fp64 two-path GEMM; weight quantization untimed",
            "seconds": elapsed, "host_cpus": len(os.sched_getaffinity(0)), "cpu": platform.processor() or None}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-rows", type=int, default=128)
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              f"(the layer shards by rows or columns without kernel changes; see the design notes)",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2606_26587_amd import sharq as S
    from paper_2606_26587_amd import synth

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    stream = torch.cuda.current_stream()

    def to_dev(u16):
        return torch.from_numpy(np.ascontiguousarray(u16).view(np.int16)).view(torch.bfloat16).to(dev)

    layers = []
    for name, (K, N, norm) in synth.LLAMA_LINEARS.items():
        xs = [to_dev(synth.activations(T_TOKENS, K, seed=s)) for s in range(N_INPUT_SETS)]
        g = to_dev(synth.gamma(K, seed=0)) if norm else None
        w = S.sharq_quantize_weight(to_dev(synth.weight(N, K, seed=0)))
        acts = [S.alloc_act(T_TOKENS, K, 2, 4, "mx", dev) for _ in range(N_INPUT_SETS)]
        ys = [torch.empty((T_TOKENS, N), dtype=torch.bfloat16, device=dev) for _ in range(N_INPUT_SETS)]
        layers.append(dict(name=name, K=K, N=N, norm=norm, xs=xs, g=g, w=w, acts=acts, ys=ys))
    torch.cuda.synchronize()
    log(f"[bench] set up {len(layers)} linears, M={T_TOKENS}")

    def step(i, ev=None):
        j = i % N_INPUT_SETS
        for li, L in enumerate(layers):
            if ev is not None:
                ev[li][0].record(stream)
            S.sharq_prepare(L["xs"][j], L["g"], synth.LLAMA_EPS, 2, 4, "mx", out=L["acts"][j], stream=stream)
            if ev is not None:
                ev[li][1].record(stream)
            S.sharq_linear(L["acts"][j], L["w"], out=L["ys"][j], stream=stream)
            if ev is not None:
                ev[li][2].record(stream)

    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    log(f"[bench] warmup {args.warmup} done")

    # timed region: exactly K steps, synchronized on both sides; per-kernel
    # HIP events are recorded on the launch stream inside the same region
    evs = [[[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in layers] for _ in range(args.steps)]
    t_start, t_end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for i in range(args.steps):
        step(i, evs[i])
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps
    log(f"[bench] timed {args.steps} steps: {ms_step:.4f} ms/step (wall {wall * 1e3 / args.steps:.4f} ms/step)")

    per = []
    flops_step = 0.0
    t_gemm = t_prep = 0.0
    bytes_prep = 0.0
    for li, L in enumerate(layers):
        prep_ms = float(np.mean([evs[i][li][0].elapsed_time(evs[i][li][1]) for i in range(args.steps)]))
        gemm_ms = float(np.mean([evs[i][li][1].elapsed_time(evs[i][li][2]) for i in range(args.steps)]))
        f = gemm_flops(T_TOKENS, L["N"], L["K"])
        b = prep_bytes(T_TOKENS, L["K"], L["norm"])
        flops_step += f
        t_gemm += gemm_ms
        t_prep += prep_ms
        bytes_prep += b
        per.append({"linear": L["name"], "K": L["K"], "N": L["N"], "rmsnorm": L["norm"],
                    "prep_us": prep_ms * 1e3, "prep_GBps": b / (prep_ms * 1e-3) / 1e9,
                    "gemm_us": gemm_ms * 1e3, "gemm_TFLOPs": f / (gemm_ms * 1e-3) / 1e12})
    value = flops_step / (ms_step * 1e-3) / 1e12
    gemm_tf = flops_step / (t_gemm * 1e-3) / 1e12
    prep_gbps = bytes_prep / (t_prep * 1e-3) / 1e9
    for p in per:
        log(f"[bench] {p['linear']:8s} prep {p['prep_us']:8.2f} us {p['prep_GBps']:8.1f} GB/s | "
            f"gemm {p['gemm_us']:8.2f} us {p['gemm_TFLOPs']:8.1f} TFLOP/s")

    out = {
        "metric": METRIC, "value": value, "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": ms_step, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "mxfp4", "data": "synthetic",
        "config": {"workload": "Llama-3.1-8B prefill linears qkv (K4096,N6144,RMSNorm), gate_up (K4096,N28672,"
                               "RMSNorm), down (K14336,N4096); M=2048 tokens; 2:4 backbone; MXFP4; bf16 out",
                   "tokens": T_TOKENS, "pattern": "2:4", "format": "MXFP4",
                   "flops_per_step": flops_step, "flops_counting": "4*M*N*K per linear (two dense-executed FP4 GEMMs)"},
        "roofline": {"bound": "mfma", "kernel": "k_linear_mx (two-path FP4 GEMM)", "achieved": gemm_tf,
                     "peak": PEAK_FP4_TFLOPS, "unit": "TFLOP/s", "frac": gemm_tf / PEAK_FP4_TFLOPS, "traffic": None},
        "prep": {"bound": "hbm", "kernel": "k_prep_mx_* (fused preparation)", "achieved": prep_gbps,
                 "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": prep_gbps / PEAK_HBM_GBPS},
        "per_linear": per,
        "wall_ms_per_step": wall * 1e3 / args.steps,
    }
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle on a bounded sample ...")
        out["cpu_baseline"] = cpu_baseline(args.cpu_rows)
        log(f"[bench] cpu oracle: {out['cpu_baseline']['value']:.4f} TFLOP/s in {out['cpu_baseline']['seconds']:.1f} s")
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
