"""Reference products and comparison metrics.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Covers
  * the model-dtype product of Sec. 5.3: y = x W_hat^T with the continuous
    reconstruction of eq. cubic as the semantic reference, evaluated in float64
    with x widened exactly from its activation dtype;
  * the comparison metric used for floating-point outputs.  The final cast to
    a 16-bit output dtype is itself a rounding of up to half an output ulp, so
    the metric excuses that half ulp once and measures what remains relative
    to the largest reference magnitude:

        eps_comp = max_i max(0, |y_gpu_i - y_ref_i| - ulp_i / 2) / max_i |y_ref_i|

    with ulp_i the larger of the output-dtype ulps at y_ref_i and y_gpu_i.
"""
from __future__ import annotations

import numpy as np

from .format import decode


def gemm_model_dtype(x, codes, bits: int, group: int, scale, a_bits, b_bits) -> np.ndarray:
    """y = x W_hat^T in float64 (Sec. 5.3; W_hat from eq. cubic)."""
    w = decode(codes, bits, group, scale, a_bits, b_bits)
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    return x @ w.T


def _ulp(v, mant_bits: int, min_exp: int) -> np.ndarray:
    """Spacing of a binary format with ``mant_bits`` stored mantissa bits."""
    av = np.abs(np.asarray(v, dtype=np.float64))
    e = np.floor(np.log2(np.where(av > 0, av, 1.0)))
    e = np.maximum(e, min_exp)
    return np.ldexp(1.0, (e - mant_bits).astype(np.int64))


def ulp_of(v, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return _ulp(v, 7, -126)
    if dtype == "fp16":
        return _ulp(v, 10, -14)
    if dtype == "fp32":
        return _ulp(v, 23, -126)
    raise ValueError(dtype)


def eps_comp(y_gpu, y_ref, out_dtype: str) -> float:
    """Computation error beyond the final output rounding (see module doc)."""
    y_gpu = np.asarray(y_gpu, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    denom = np.max(np.abs(y_ref)) if y_ref.size else 0.0
    if denom == 0:
        return float(np.max(np.abs(y_gpu))) if y_gpu.size else 0.0
    half = 0.5 * np.maximum(ulp_of(y_ref, out_dtype), ulp_of(y_gpu, out_dtype))
    excess = np.maximum(0.0, np.abs(y_gpu - y_ref) - half)
    return float(np.max(excess) / denom)


def rel_rms(y_gpu, y_ref) -> float:
    y_gpu = np.asarray(y_gpu, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    den = np.linalg.norm(y_ref)
    return float(np.linalg.norm(y_gpu - y_ref) / den) if den > 0 else float(np.linalg.norm(y_gpu))
