"""Shared seeded test cases: oracle-fitted weights and their oracle references.

Inputs come from ``workloads`` (seeded draws) and ``oracle`` (fit, pack,
references); nothing here calls the HIP library.
"""
from __future__ import annotations

import functools
import sys

import numpy as np

from oracle import a8 as A8
from oracle import fit as FIT
from oracle import format as F
from oracle import ref as R
from workloads import bf16_bits_to_f32, small_act, small_weight, to_f16_bits


def say(*args):
    """Name the case before a GPU step (flushed, so a crash still shows it)."""
    print("[case]", *args, flush=True)
    sys.stdout.flush()


@functools.lru_cache(maxsize=None)
def fitted(seed: int, n: int, k: int, bits: int, group: int, law: str = "laplace", int_only: bool = False):
    w = small_weight(seed, n, k, law)
    if int_only:
        r = FIT.fit(w, bits, group, candidates=(np.array([1.0]), np.array([0.0])), refine_steps=())
    else:
        r = FIT.fit(w, bits, group)
    return r


def act(seed: int, m: int, k: int, dtype: str = "bf16", outliers: bool = True):
    """Activation bit patterns and their exact float64 values."""
    bits = small_act(seed, m, k, outliers)
    vals = bf16_bits_to_f32(bits).astype(np.float64)
    if dtype == "fp16":
        bits = to_f16_bits(vals)
        vals = F.f16_bits_to_f64(bits)
    return bits, vals


def ref_model_dtype(x_vals, r, bits: int, group: int):
    return R.gemm_model_dtype(x_vals, r.codes, bits, group, r.scale, r.a_bits, r.b_bits)


def ref_a8(x_vals, r, bits: int, group: int):
    x8, dx = A8.quantize_act(x_vals)
    y, p = A8.gemm_a8(x8, dx, r.codes, bits, group, r.scale, r.a_bits, r.b_bits)
    return x8, dx, y, p


@functools.lru_cache(maxsize=None)
def near_tie_shapes(bits: int, count: int = 64, seed: int = 77):
    """FP16 shape pairs (a, b), strictly admissible, for which some interior
    carrier value 127 q(i/M) lies within 3e-4 of a half-integer (the closest
    found first).  Exact values come from the oracle's rational carrier table;
    the screening uses float64."""
    m = F.max_code(bits)
    rng = np.random.default_rng(seed)
    a = F.f16_bits_to_f64(to_f16_bits(rng.uniform(0.05, 1.6, 400_000)))
    b = F.f16_bits_to_f64(to_f16_bits(rng.uniform(-1.3, 0.5, 400_000)))
    ok = F.admissible_strict(a, b)
    a, b = a[ok], b[ok]
    t = np.arange(1, m) / m
    v = 127.0 * F.q_curve(t[None, :], a[:, None], b[:, None])
    d = np.abs(np.abs(v - np.floor(v)) - 0.5).min(axis=1)
    order = np.argsort(d)
    picked, seen = [], set()
    for i in order:
        if d[i] > 3e-4 or len(picked) == count:
            break
        key = (int(to_f16_bits(a[i])), int(to_f16_bits(b[i])))
        if key not in seen:
            seen.add(key)
            picked.append(key)
    return picked


def carrier_probe(bits: int, group: int, seed: int = 5):
    """Weights whose rows use near-tie shapes with unit scales and every code,
    plus INT8 activations: y = sum_g P_g is an exact integer in FP32."""
    shapes = near_tie_shapes(bits)
    m = F.max_code(bits)
    n = len(shapes)
    ng = 2
    k = group * ng
    rng = np.random.default_rng(seed)
    pool = np.array([c for c in range(-m, m + 1)], dtype=np.int64) if bits > 1 else np.array([-1, 1])
    codes = pool[rng.integers(0, len(pool), size=(n, k))].astype(np.int8)
    a = np.zeros((n, ng), np.uint16)
    b = np.zeros((n, ng), np.uint16)
    for r in range(n):
        for g in range(ng):
            a[r, g], b[r, g] = shapes[(r + 7 * g) % n]
    s = np.ones((n, ng), np.float32)
    x8 = rng.integers(-127, 128, size=(1, k)).astype(np.int8)
    dx = np.full(1, 127.0, np.float32)
    _, p = A8.gemm_a8(x8, dx, codes, bits, group, s, a, b)
    return codes, s, a, b, x8, dx, p
