"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module only draws random numbers and rounds them to bf16; it holds none of
SharQ's arithmetic.  Streams come from NumPy's PCG64 through
SeedSequence(seed).spawn(4): X, gamma, W and router logits.

Activation recipe (stands in for LLM activations; the paper evaluates on real
Llama/Qwen activations, which are not available here):
  * X ~ N(0, 1);
  * round(0.005 K) outlier channels, drawn without replacement, multiplied by
    U(20, 100);
  * one "massive activation": token 0 multiplied by 1000 on 2 channels;
  * gamma = 1 + N(0, 0.1);  W ~ N(0, 0.02).
The small single-linear case instead scales the fixed channels 3 and 77 by 50.
"""

from __future__ import annotations

import numpy as np


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest even (finite inputs)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_bits_to_f32(u16: np.ndarray) -> np.ndarray:
    return (np.asarray(u16, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _streams(seed: int):
    return [np.random.Generator(np.random.PCG64(s)) for s in np.random.SeedSequence(seed).spawn(4)]


def activations(T: int, K: int, seed: int = 0, fixed_outliers=None, outlier_scale: float = 50.0,
                massive: bool = True) -> np.ndarray:
    """Outlier-bearing activation rows X[T, K] as bf16 bits."""
    rx = _streams(seed)[0]
    x = rx.standard_normal((T, K), dtype=np.float32)
    if fixed_outliers is not None:
        for c in fixed_outliers:
            x[:, c] *= np.float32(outlier_scale)
    else:
        n_out = int(round(0.005 * K))
        if n_out > 0:
            ch = rx.choice(K, size=n_out, replace=False)
            x[:, ch] *= rx.uniform(20.0, 100.0, size=n_out).astype(np.float32)[None, :]
        if massive and T > 0 and K >= 2:
            ch2 = rx.choice(K, size=2, replace=False)
            x[0, ch2] *= np.float32(1000.0)
    return f32_to_bf16_bits(x)


def gamma(K: int, seed: int = 0) -> np.ndarray:
    rg = _streams(seed)[1]
    return f32_to_bf16_bits((1.0 + 0.1 * rg.standard_normal(K)).astype(np.float32))


def weight(N: int, K: int, seed: int = 0) -> np.ndarray:
    rw = _streams(seed)[2]
    return f32_to_bf16_bits((0.02 * rw.standard_normal((N, K))).astype(np.float32))


def router_topk(T: int, E: int, topk: int, seed: int = 0):
    """Top-k routing from N(0,1) router logits (ties -> lower expert id).

    Returns (row_index, expert_offsets): the (token, slot) pairs sorted by
    expert; row_index[i] is the token of pair i, expert_offsets[e] the first
    pair routed to expert e (E + 1 entries).
    """
    rr = _streams(seed)[3]
    logits = rr.standard_normal((T, E)).astype(np.float32)
    # stable sort on -logit keeps the lower expert id first among equal logits
    order = np.argsort(-logits, axis=1, kind="stable")[:, :topk]
    experts = order.reshape(-1)
    tokens = np.repeat(np.arange(T), topk)
    perm = np.argsort(experts, kind="stable")
    row_index = tokens[perm].astype(np.int32)
    counts = np.bincount(experts, minlength=E)
    offsets = np.zeros(E + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(counts)
    return row_index, offsets


def tiny_case(seed: int = 0):
    """The small single linear: X[8,128] with channels 3 and 77 x50, W[64,128]."""
    return {"x": activations(8, 128, seed, fixed_outliers=(3, 77), outlier_scale=50.0, massive=False),
            "gamma": gamma(128, seed), "w": weight(64, 128, seed), "eps": 1e-6, "n": 2, "m": 4}


#: Llama-3.1-8B linear shapes (K, N, has RMSNorm) at M = 2048 tokens.
LLAMA_LINEARS = {
    "qkv": (4096, 6144, True),
    "gate_up": (4096, 28672, True),
    "down": (14336, 4096, False),
}
LLAMA_EPS = 1e-5
#: Qwen2.5-7B linear shapes (NVFP4 case) at M = 4096 tokens.
QWEN_LINEARS = {
    "gate_up": (3584, 37888, True),
    "down": (18944, 3584, False),
}
#: Qwen3-30B-A3B MoE shapes: hidden 2048, 128 experts, expert intermediate 768, top-8.
MOE = {"hidden": 2048, "experts": 128, "inter": 768, "topk": 8, "tokens": 4096}
