"""Seeded synthetic inputs shared by the oracle-side tests and the GPU path.

This module only draws random numbers and rounds them to the storage dtypes
(float32 weights, bfloat16 / float16 activation bit patterns).  It holds none
of the CubicQuant arithmetic: no packing, no level function, no fitting, no
quantizer.  Every generator uses numpy's PCG64 with its own seed, draws in
float64 and rounds once.

The workloads are the layer shapes and value laws of the benchmark
configurations:
  * ``gemv_4k``    M=1, K=N=4096; x ~ N(0,1) (seed 0), W ~ N(0, 0.02^2) (seed 1).
  * ``llama8b``    Llama-3-8B-shaped decode layers (K, N) in
    {(4096, 6144) QKV, (4096, 4096) O, (4096, 28672) gate+up, (14336, 4096) down},
    M in {1, 4, 16}; W ~ Laplace(0, 0.014) with ceil(0.01 K) input channels
    scaled x8; x ~ N(0,1) times a per-token factor ~ U[0.5, 4].
  * ``sweep``      M=1, K=N=8192, W ~ N(0, 0.015^2), every B x G.
  * ``crossover``  K=8192, N=28672, M in {1 .. 8192}; W ~ Student-t(5) scaled to
    std 0.02; x ~ N(0,1) with 0.5% of entries scaled x20.
  * ``prefill70b`` M in {2048, 8192}, (K, N) in {(8192, 28672), (28672, 8192),
    (8192, 10240)}; W ~ Laplace(0, 0.01) times a per-row factor log-uniform in
    [0.5, 2]; x ~ N(0,1).
Seeds: for workload number c (1..5) tensor t uses 1000*c + t, except the first
workload whose x uses seed 0 and W seed 1.  The weights of the larger
workloads are drawn row by row, each row from its own generator seeded by
(tensor seed, row index), so that a sample of rows can be drawn (and fitted)
without the whole matrix.
"""
from __future__ import annotations

import math

import numpy as np

LLAMA8B_LAYERS = (("qkv", 4096, 6144), ("o_proj", 4096, 4096),
                  ("gate_up", 4096, 28672), ("down", 14336, 4096))
PREFILL70B_SHAPES = ((8192, 28672), (28672, 8192), (8192, 10240))
CROSSOVER_M = (1, 2, 8, 32, 128, 512, 2048, 8192)


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def to_f32(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float32)


def to_bf16_bits(x) -> np.ndarray:
    """Round float64 -> float32 -> bfloat16 (nearest even), return uint16 bits."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float64).astype(np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16).astype(np.uint16)
    nan = np.isnan(f)
    if np.any(nan):
        r = np.where(nan, np.uint16(0x7FC0), r)
    return r


def to_f16_bits(x) -> np.ndarray:
    return np.asarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


def bf16_bits_to_f32(bits) -> np.ndarray:
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


# ---------------------------------------------------------------- value laws


def normal(seed: int, shape, std: float = 1.0) -> np.ndarray:
    return rng(seed).standard_normal(shape) * std


def laplace(seed: int, shape, b: float) -> np.ndarray:
    return rng(seed).laplace(0.0, b, shape)


def student_t(seed: int, shape, nu: float, std: float) -> np.ndarray:
    return rng(seed).standard_t(nu, shape) * (std / math.sqrt(nu / (nu - 2.0)))


# ---------------------------------------------------------------- workloads


def gemv_4k():
    """(x bf16 bits [1, 4096], W float32 [4096, 4096])."""
    x = to_bf16_bits(normal(0, (1, 4096)))
    w = to_f32(normal(1, (4096, 4096), 0.02))
    return x, w


def row_rng(seed: int, row: int) -> np.random.Generator:
    """Generator of one weight row: PCG64 seeded by the pair (tensor seed, row),
    so that any subset of rows of a large matrix can be drawn on its own."""
    return np.random.Generator(np.random.PCG64([seed, int(row)]))


def _rows(rows, n: int) -> np.ndarray:
    r = np.arange(n) if rows is None else np.asarray(rows, dtype=np.int64)
    if r.size and (r.min() < 0 or r.max() >= n):
        raise IndexError("row outside the matrix")
    return r


def llama8b_outlier_cols(layer: int, k: int) -> np.ndarray:
    """The ceil(0.01 K) input channels of a decode layer scaled x8."""
    return rng(2001 + 2 * layer).choice(k, size=math.ceil(0.01 * k), replace=False)


def llama8b_weight(layer: int, k: int, n: int, rows=None) -> np.ndarray:
    """Rows `rows` (default all) of the Laplace(0, 0.014) weights [N, K] of a
    decode layer, with ceil(0.01 K) input channels x8."""
    r = _rows(rows, n)
    w = np.empty((r.size, k))
    for i, row in enumerate(r):
        w[i] = row_rng(2000 + 2 * layer, row).laplace(0.0, 0.014, k)
    w[:, llama8b_outlier_cols(layer, k)] *= 8.0
    return to_f32(w)


def llama8b_act(m: int, k: int, seed_offset: int = 0) -> np.ndarray:
    """bf16 bits [M, K]: N(0,1) rows times a per-token factor ~ U[0.5, 4]."""
    x = normal(2100 + seed_offset, (m, k))
    u = rng(2101 + seed_offset).uniform(0.5, 4.0, (m, 1))
    return to_bf16_bits(x * u)


def sweep_weight(k: int = 8192, n: int = 8192, rows=None) -> np.ndarray:
    """Rows of the N(0, 0.015^2) weights of the bit-width / group sweep."""
    r = _rows(rows, n)
    w = np.empty((r.size, k))
    for i, row in enumerate(r):
        w[i] = row_rng(3001, row).standard_normal(k) * 0.015
    return to_f32(w)


def sweep_act(k: int = 8192) -> np.ndarray:
    return to_bf16_bits(normal(3002, (1, k)))


def crossover_weight(k: int = 8192, n: int = 28672, rows=None) -> np.ndarray:
    """Rows of the Student-t(5) weights scaled to std 0.02 (crossover shape)."""
    r = _rows(rows, n)
    w = np.empty((r.size, k))
    for i, row in enumerate(r):
        w[i] = row_rng(4001, row).standard_t(5.0, k) * (0.02 / math.sqrt(5.0 / 3.0))
    return to_f32(w)


def crossover_act(m: int, k: int = 8192) -> np.ndarray:
    x = normal(4002, (m, k))
    mask = rng(4003).random((m, k)) < 0.005
    x[mask] *= 20.0
    return to_bf16_bits(x)


def prefill70b_row_multipliers(n: int, seed_offset: int = 0) -> np.ndarray:
    """Per-output-row std multipliers, log-uniform in [0.5, 2]."""
    return np.exp(rng(5002 + seed_offset).uniform(math.log(0.5), math.log(2.0), n))


def prefill70b_weight(k: int, n: int, seed_offset: int = 0, rows=None) -> np.ndarray:
    """Rows of the Laplace(0, 0.01) weights times their row multiplier."""
    r = _rows(rows, n)
    mult = prefill70b_row_multipliers(n, seed_offset)[r]
    w = np.empty((r.size, k))
    for i, row in enumerate(r):
        w[i] = row_rng(5001 + seed_offset, row).laplace(0.0, 0.01, k) * mult[i]
    return to_f32(w)


def prefill70b_act(m: int, k: int) -> np.ndarray:
    return to_bf16_bits(normal(5003, (m, k)))


def small_weight(seed: int, n: int, k: int, law: str = "laplace") -> np.ndarray:
    """Small test matrices with the same laws as the workloads."""
    if law == "laplace":
        w = laplace(seed, (n, k), 0.014)
        cols = rng(seed + 1).choice(k, size=max(1, math.ceil(0.01 * k)), replace=False)
        w[:, cols] *= 8.0
    elif law == "normal":
        w = normal(seed, (n, k), 0.02)
    elif law == "student":
        w = student_t(seed, (n, k), 5.0, 0.02)
    else:
        raise ValueError(law)
    return to_f32(w)


def small_act(seed: int, m: int, k: int, outliers: bool = True) -> np.ndarray:
    x = normal(seed, (m, k)) * rng(seed + 1).uniform(0.5, 4.0, (m, 1))
    if outliers:
        mask = rng(seed + 2).random((m, k)) < 0.005
        x[mask] *= 20.0
    return to_bf16_bits(x)


# ---------------------------------------------------------------- packed-representation stand-in
#
# Shape pairs printed in the paper's population tables (Gaussian / Laplace
# optima, Sec. 3.3), used as fixed, known-monotone curve shapes.
PRINTED_SHAPES = ((1.0, 0.0), (0.7932, -0.3847), (0.5203, -0.2936), (0.8517, -0.1852),
                  (0.6216, -0.1495), (0.7510, -0.5253), (0.4603, -0.3881))


def synthetic_representation(seed: int, n: int, k: int, bits: int, group: int, scale_center: float = 0.05,
                             block_rows: int | None = None):
    """Random stand-in for a quantized matrix: codes drawn from a rounded
    Laplace law clipped to [-M, M], lognormal FP32 scales and shapes taken from
    PRINTED_SHAPES.  Kernel timing does not depend on the values, only on the
    layout, so this serves timing runs that must not call the oracle.  With
    block_rows, only that many rows are drawn and repeated down the matrix
    (a faster stand-in for large timing matrices)."""
    if block_rows is not None and block_rows < n:
        parts = synthetic_representation(seed, block_rows, k, bits, group, scale_center)
        reps = -(-n // block_rows)
        return tuple(np.ascontiguousarray(np.tile(p, (reps, 1))[:n]) for p in parts)
    g = rng(seed)
    m = 1 if bits == 1 else (1 << (bits - 1)) - 1
    if bits == 1:
        codes = np.where(g.random((n, k)) < 0.5, -1, 1).astype(np.int8)
    else:
        raw = np.rint(g.laplace(0.0, max(m / 3.0, 0.5), (n, k)))
        codes = np.clip(raw, -m, m).astype(np.int8)
    ng = k // group
    scale = (scale_center * np.exp(0.3 * g.standard_normal((n, ng)))).astype(np.float32)
    pick = g.integers(0, len(PRINTED_SHAPES), (n, ng))
    shapes = np.array(PRINTED_SHAPES)
    a_bits = to_f16_bits(shapes[pick, 0])
    b_bits = to_f16_bits(shapes[pick, 1])
    return codes, scale, a_bits, b_bits


# ---------------------------------------------------------------- routed (mixture-of-experts) inputs

# Mixtral-8x7B-shaped expert layers (K, N) with 8 experts, top-2 routing.
MOE_LAYERS = (("expert_gate_up", 4096, 28672), ("expert_down", 14336, 4096))
MOE_EXPERTS = 8
MOE_TOPK = 2


def route_map(seed: int, tokens: int, experts: int, topk: int, skew: float = 1.0):
    """Synthetic route map: every token picks topk distinct experts, drawn
    with Zipf-like popularity 1 / (rank + 1)^skew over a seeded permutation of
    the experts (so some experts are busier than others).  Returns int32
    (route_token, route_expert), token-major."""
    g = rng(seed)
    pop = 1.0 / np.arange(1, experts + 1) ** skew
    perm = g.permutation(experts)
    p = np.empty(experts)
    p[perm] = pop / pop.sum()
    toks, exps = [], []
    for t in range(tokens):
        picks = g.choice(experts, size=min(topk, experts), replace=False, p=p)
        toks.extend([t] * len(picks))
        exps.extend(picks.tolist())
    return np.asarray(toks, dtype=np.int32), np.asarray(exps, dtype=np.int32)
