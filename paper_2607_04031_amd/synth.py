"""Seeded synthetic inputs for the tile-major GEMM path.

This module only draws numbers.  It holds none of the method's arithmetic
(no layout, no GEMM, no amplification count), so that the CPU oracle and the
HIP path can be fed the very same bytes.  Everything is numpy PCG64
(``default_rng(seed)``), float32 normal draws scaled by sigma, then rounded to
bfloat16 with round-to-nearest-even.  Weights are generated ROW-MAJOR
``[N, K]`` (the ``nn.Linear.weight`` orientation); the tile-major copy is made
by the library's repack.

Workload shapes follow the paper's evaluation models (Section 6.2): the dense
FFN/attention projections of a Llama-3.1-70B-class model and the MoE experts
and attention of a Qwen-3-30B-A3B-class model.  No model weights or traces are
used: the values are random, only the shapes and distributions are real.
"""
from __future__ import annotations

import numpy as np

# --------------------------------------------------------------------------
# bf16 bit handling (input generation only)
# --------------------------------------------------------------------------


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round-to-nearest-even.

    Inputs here are finite normal draws; NaN/Inf need no special case."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    return ((u + bias) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(h: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(h, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def normal_bf16(shape, seed: int, sigma: float = 1.0) -> np.ndarray:
    """bf16 bits of sigma * N(0, 1) draws, PCG64(seed), float32 draws."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        x *= np.float32(sigma)
    return f32_to_bf16_bits(x)


def small_int_bf16(shape, seed: int, lo: int = -4, hi: int = 4) -> np.ndarray:
    """bf16 bits of uniform integers in [lo, hi] (exactly representable)."""
    rng = np.random.default_rng(seed)
    x = rng.integers(lo, hi + 1, size=shape).astype(np.float32)
    return f32_to_bf16_bits(x)


def one_hot_bf16(M: int, K: int, seed: int) -> tuple[np.ndarray, np.ndarray]:
    """Rows A[m] = e_{k_m} (value 1.0), k_m drawn uniformly.  Returns (bits, k_m)."""
    rng = np.random.default_rng(seed)
    ks = rng.integers(0, K, size=M)
    A = np.zeros((M, K), dtype=np.float32)
    A[np.arange(M), ks] = 1.0
    return f32_to_bf16_bits(A), ks


def random_bytes(nbytes: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(0, 256, size=nbytes, dtype=np.uint8)


# --------------------------------------------------------------------------
# Workloads (shapes and seeds)
# --------------------------------------------------------------------------

W_SIGMA = 0.02           # weights ~ N(0, 0.02^2)
A_SIGMA = 1.0            # activations ~ N(0, 1)

# Llama-3.1-70B-class projections, weight stored [N, K] (out, in).
LLAMA70B = [
    ("qkv", 10240, 8192),
    ("o", 8192, 8192),
    ("gate_up", 57344, 8192),
    ("down", 8192, 28672),
]
LLAMA_DECODE_M = (1, 8, 32)
LLAMA_PREFILL_M = 2048


def llama_weight_seed(i: int) -> int:
    return 10 + i


def llama_decode_act_seed(i: int, M: int) -> int:
    return 20 + i + 100 * M


def llama_prefill_act_seed(i: int, M: int = LLAMA_PREFILL_M) -> int:
    return 30 + i if M == LLAMA_PREFILL_M else 30 + i + 100 * M


# Qwen-3-30B-A3B-class MoE layer.
QWEN_EXPERTS = 128
QWEN_TOPK = 8
QWEN_HIDDEN = 2048
QWEN_GATE_UP = (1536, 2048)      # [N, K]
QWEN_DOWN = (2048, 768)          # [N, K]
QWEN_ATTN = [("q", 4096, 2048), ("k", 512, 2048), ("v", 512, 2048), ("o", 2048, 4096)]
QWEN_TOKENS = 64


def qwen_gate_up_seed(e: int) -> int:
    return 1000 + e


def qwen_down_seed(e: int) -> int:
    return 2000 + e


def moe_routing(M: int = QWEN_TOKENS, E: int = QWEN_EXPERTS, topk: int = QWEN_TOPK,
                seed: int = 42) -> np.ndarray:
    """Per token, ``topk`` distinct experts drawn uniformly without replacement,
    token by token from one PCG64(seed) stream.  Returns int64 [M, topk]."""
    rng = np.random.default_rng(seed)
    return np.stack([rng.choice(E, topk, replace=False) for _ in range(M)]).astype(np.int64)


def tokens_per_expert(routing: np.ndarray, E: int = QWEN_EXPERTS) -> list[np.ndarray]:
    """Token indices routed to each expert, ascending."""
    out = []
    for e in range(E):
        out.append(np.nonzero((routing == e).any(axis=1))[0].astype(np.int64))
    return out


def qwen_attn_seed(i: int) -> int:
    """Seed of attention projection QWEN_ATTN[i] (q, k, v, o)."""
    return 3000 + i


QWEN_SEED_HIDDEN = 3      # [64, 2048] hidden states: input of q, k, v and of the experts' gate+up
QWEN_SEED_ATTN_O_IN = 5   # [64, 4096] attention output: input of o
QWEN_SEED_DOWN_IN = 4     # [sum of tokens per expert, 768] input of the experts' down GEMMs


def moe_tables(routing: np.ndarray, E: int = QWEN_EXPERTS) -> tuple[np.ndarray, np.ndarray]:
    """Grouped-launch tables for a routing: int32 offsets [E + 1] (rows of
    expert e are offsets[e] .. offsets[e+1] - 1) and int32 token ids, the
    tokens of each expert in ascending order, experts one after another."""
    tok = tokens_per_expert(routing, E)
    offsets = np.zeros(E + 1, dtype=np.int32)
    offsets[1:] = np.cumsum([len(t) for t in tok])
    ids = np.concatenate(tok).astype(np.int32) if offsets[-1] else np.zeros(0, dtype=np.int32)
    return offsets, ids


def quantize_e4m3(w: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    """Per-output-channel FP8 (OCP E4M3) weights for a float32 [N, K] array:
    scales[n] = max_k |w[n, k]| / 448 (448 = the largest E4M3 value) and the
    bytes of w / scales rounded to nearest even by torch's float8_e4m3fn
    conversion.  Returns (uint8 [N, K], float32 [N])."""
    import torch
    w = np.ascontiguousarray(w, dtype=np.float32)
    amax = np.abs(w).max(axis=1)
    scales = np.where(amax > 0, amax / np.float32(448.0), np.float32(1.0)).astype(np.float32)
    q = torch.from_numpy(w / scales[:, None]).to(torch.float8_e4m3fn)
    return q.view(torch.uint8).numpy().copy(), scales


def fp8_weights(shape, seed: int, sigma: float = W_SIGMA) -> tuple[np.ndarray, np.ndarray]:
    """FP8 weights of the normal_bf16 draw with the same seed (float32 draws,
    before bf16 rounding), per-channel scaled."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if sigma != 1.0:
        x *= np.float32(sigma)
    return quantize_e4m3(x)
