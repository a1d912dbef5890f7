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
