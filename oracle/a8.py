"""Dynamic-A8 execution semantics, restated in exact arithmetic.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

Covers
  * the per-row activation scale and INT8 activation carrier of Sec. 5.4
    (eq. a8-activation-scale, eq. a8-activation-quantization), with
    round-half-away-from-zero and clipping to [-127, 127];
  * the INT8 weight carrier of Sec. 4.3 (eq. carrier, eq. carrier-grid) with
    round-to-nearest-even (Appendix A, item 7);
  * the INT32 group partials, the FP32 group rescale and the cross-group sum of
    Sec. 5.4 (eq. a8-output) and the INT32 bound (eq. a8-int32-bound).

Readings taken where the paper leaves a choice open:
  * the safeguard epsilon is fl32(1e-10);
  * d_x = fl32(xbar / 127) and v_j = fl32(x_j / d_x) are IEEE binary32
    divisions.  They are computed here in float64 and rounded once to binary32,
    which equals the correctly rounded binary32 quotient because
    53 >= 2*24 + 2 (double rounding is innocuous for division);
  * the carrier is RNE of the exact rational 127*q(|k|/M) built from the
    serialized FP16 shape values (fractions.Fraction, no floating point).
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

from .format import f16_bits_to_f64, max_code

EPS = float(np.float32(1e-10))


def round_half_away(v) -> np.ndarray:
    """Nearest integer, halfway cases away from zero."""
    v = np.asarray(v, dtype=np.float64)
    return np.sign(v) * np.floor(np.abs(v) + 0.5)


def quantize_act(x) -> tuple[np.ndarray, np.ndarray]:
    """Per-row dynamic INT8 quantization (eq. a8-activation-scale/-quantization).

    x: float64 [M, K] holding values exactly representable in the activation
    dtype.  Returns x8 int8 [M, K] and d_x float32 [M].
    """
    x = np.atleast_2d(np.asarray(x, dtype=np.float64))
    xbar = np.maximum(np.max(np.abs(x), axis=1), EPS)
    d = (xbar / 127.0).astype(np.float32).astype(np.float64)
    v = (x / d[:, None]).astype(np.float32).astype(np.float64)
    x8 = np.clip(round_half_away(v), -127, 127).astype(np.int8)
    return x8, d.astype(np.float32)


def _rne_fraction(v: Fraction) -> int:
    """Round a rational to the nearest integer, ties to even."""
    return round(v)  # Fraction.__round__ with no digits rounds half to even


def carrier_table(bits: int, a_bits: int, b_bits: int) -> list:
    """r(i) = RNE(127 q(i/M)) for magnitudes i = 0..M (eq. carrier).

    q is evaluated exactly from the FP16 values a, b (c = 1 - a - b).
    W1 uses the single magnitude 1 with r = 127.
    """
    if bits == 1:
        return [0, 127]
    m = max_code(bits)
    a = Fraction(float(f16_bits_to_f64(a_bits)))
    b = Fraction(float(f16_bits_to_f64(b_bits)))
    c = 1 - a - b
    out = []
    for i in range(m + 1):
        t = Fraction(i, m)
        q = t * (a + t * (b + t * c))
        out.append(_rne_fraction(127 * q))
    return out


def carriers(codes, bits: int, group: int, a_bits, b_bits) -> np.ndarray:
    """Signed INT8 weight carriers r(k) = sign(k) RNE(127 q(|k|/M)) per weight."""
    codes = np.atleast_2d(np.asarray(codes, dtype=np.int64))
    n, k = codes.shape
    ng = k // group
    a_bits = np.asarray(a_bits, dtype=np.uint16).reshape(n, ng)
    b_bits = np.asarray(b_bits, dtype=np.uint16).reshape(n, ng)
    out = np.zeros((n, k), dtype=np.int64)
    cache: dict = {}
    for r in range(n):
        for g in range(ng):
            key = (int(a_bits[r, g]), int(b_bits[r, g]))
            tab = cache.get(key)
            if tab is None:
                tab = np.array(carrier_table(bits, *key), dtype=np.int64)
                cache[key] = tab
            cg = codes[r, g * group:(g + 1) * group]
            if bits == 1:
                out[r, g * group:(g + 1) * group] = cg * 127
            else:
                out[r, g * group:(g + 1) * group] = np.sign(cg) * tab[np.abs(cg)]
    return out


def group_partials(x8, r, group: int) -> np.ndarray:
    """P_g[m, n, g] = sum over j in group g of x8[m, j] r[n, j] (exact int64)."""
    x8 = np.asarray(x8, dtype=np.int64)
    r = np.asarray(r, dtype=np.int64)
    mrows, k = x8.shape
    n = r.shape[0]
    ng = k // group
    xg = x8.reshape(mrows, ng, group)
    rg = r.reshape(n, ng, group)
    return np.einsum("mgj,ngj->mng", xg, rg)


def gemm_a8(x8, dx, codes, bits: int, group: int, scale, a_bits, b_bits):
    """y[m, n] = sum_g (d_m s_{n,g} / 127) P_g[m, n, g] in float64 (eq. a8-output).

    Returns (y float64 [M, N], P int64 [M, N, K/G]).
    """
    r = carriers(codes, bits, group, a_bits, b_bits)
    p = group_partials(x8, r, group)
    n = r.shape[0]
    s = np.asarray(scale, dtype=np.float32).astype(np.float64).reshape(n, -1)
    d = np.asarray(dx, dtype=np.float32).astype(np.float64)
    y = np.einsum("mng,ng->mn", p.astype(np.float64), s) * d[:, None] / 127.0
    return y, p


def int32_bound(group: int) -> int:
    """|P_g| <= G * 127^2 (eq. a8-int32-bound)."""
    return group * 127 * 127
