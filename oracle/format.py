"""CubicQuant storage format, restated from the paper in fp64/int64.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``): never imported by the
product library.

Covers
  * the signed code space of Sec. 2.1 (eq. codes): B in 1..8, M = 2^(B-1)-1,
    codes k in [-M, M]; the two's-complement pattern -2^(B-1) is reserved and
    decodes to zero; W1 is the binary {-1, +1} case with no zero;
  * the continuous row-major bitstream of Sec. 2.1 and the byte/shift
    extraction of Sec. 5.2 (eq. gpu-packed-extraction), LSB first;
  * the cubic level function of Sec. 2.2 (eq. cubic) and the reference
    decode of Appendix B;
  * the metadata geometry of Sec. 2.3: one FP32 scale and two FP16 shape values
    per [1, G] group, and the effective width B + 64/G (eq. effective-bits);
  * the closed-form monotone shape domain m(a, b) of Sec. 3.1
    (eq. shape-domain) and the storage model of Sec. 6.2
    (eq. cubic-weight-bytes, eq. cubic-bf16-compression).

Readings taken where the paper leaves a choice open:
  * W1 field value 1 means +1 and 0 means -1 (Appendix B lists the W1 levels
    in the order (-scale, +scale)).
  * Rows are byte aligned; with K % G == 0 and G*B % 8 == 0 there are no tail
    bits, and any padding bits are zero.
"""
from __future__ import annotations

import numpy as np

# ---------------------------------------------------------------- precision helpers


def f16_bits_to_f64(bits) -> np.ndarray:
    """Widen IEEE binary16 bit patterns exactly to float64."""
    return np.asarray(bits, dtype=np.uint16).view(np.float16).astype(np.float64)


def f64_to_f16_bits(x) -> np.ndarray:
    """Round float64 to binary16 (round to nearest even) and return the bits."""
    return np.asarray(x, dtype=np.float64).astype(np.float16).view(np.uint16)


def fl32(x) -> np.ndarray:
    """Round to binary32 (round to nearest even) and widen back to float64."""
    return np.asarray(x, dtype=np.float64).astype(np.float32).astype(np.float64)


def bf16_bits_to_f64(bits) -> np.ndarray:
    """Widen bfloat16 bit patterns exactly to float64."""
    b = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16
    return b.view(np.float32).astype(np.float64)


def f16_bits_to_f64_activation(bits) -> np.ndarray:
    """Widen fp16 activation bit patterns exactly to float64."""
    return f16_bits_to_f64(bits)


# ---------------------------------------------------------------- code space (Sec. 2.1)


def max_code(bits: int) -> int:
    """M = 2^(B-1) - 1 (eq. codes); for W1 the magnitude is 1."""
    if not 1 <= bits <= 8:
        raise ValueError("payload width must be in 1..8")
    return 1 if bits == 1 else (1 << (bits - 1)) - 1


def valid_codes(bits: int) -> np.ndarray:
    """All valid signed codes of width B (2^B - 1 values; W1: {-1, +1})."""
    if bits == 1:
        return np.array([-1, 1], dtype=np.int64)
    m = max_code(bits)
    return np.arange(-m, m + 1, dtype=np.int64)


def code_to_field(k, bits: int) -> np.ndarray:
    """Unsigned B-bit field stored for signed code k.

    B >= 2: two's complement, f = k mod 2^B.  W1: +1 -> 1, -1 -> 0.
    """
    k = np.asarray(k, dtype=np.int64)
    if bits == 1:
        if np.any((k != 1) & (k != -1)):
            raise ValueError("W1 codes must be -1 or +1")
        return (k > 0).astype(np.int64)
    m = max_code(bits)
    if np.any(np.abs(k) > m):
        raise ValueError("code out of range [-M, M]")
    return np.mod(k, 1 << bits)


def field_to_code(u, bits: int) -> np.ndarray:
    """Signed code for an unsigned B-bit field (Sec. 2.1, Sec. 5.2).

    B >= 2: sign-extend; the reserved pattern -2^(B-1) decodes to 0.
    W1: u -> 2u - 1.
    """
    u = np.asarray(u, dtype=np.int64)
    if bits == 1:
        return 2 * u - 1
    half = 1 << (bits - 1)
    k = np.where(u >= half, u - (1 << bits), u)
    return np.where(u == half, 0, k)


# ---------------------------------------------------------------- bitstream


def row_bytes(k: int, bits: int) -> int:
    """Bytes per packed row (rows are byte aligned, tail bits zero)."""
    return (k * bits + 7) // 8


def pack(codes, bits: int) -> np.ndarray:
    """Pack signed codes [N, K] into the continuous LSB-first bitstream.

    Field j of a row occupies stream bits [jB, jB + B); stream bit p is bit
    (p mod 8) of byte floor(p / 8) (Sec. 2.1, and the inverse of
    eq. gpu-packed-extraction).
    """
    codes = np.atleast_2d(np.asarray(codes, dtype=np.int64))
    n, k = codes.shape
    f = code_to_field(codes, bits)
    # bit b of field j goes to stream position j*B + b
    bitplanes = ((f[:, :, None] >> np.arange(bits)[None, None, :]) & 1).astype(np.uint8)
    stream = bitplanes.reshape(n, k * bits)
    pad = row_bytes(k, bits) * 8 - k * bits
    if pad:
        stream = np.concatenate([stream, np.zeros((n, pad), np.uint8)], axis=1)
    return np.packbits(stream, axis=1, bitorder="little")


def unpack_fields(packed, bits: int, k: int) -> np.ndarray:
    """Extract the unsigned fields u_j of every row (eq. gpu-packed-extraction).

    p_j = floor(jB/8), d_j = jB mod 8,
    u_j = [(byte[p_j] >> d_j) | (byte[p_j + 1] << (8 - d_j))] & (2^B - 1),
    the second byte omitted when the field does not cross a byte boundary.
    """
    packed = np.atleast_2d(np.asarray(packed, dtype=np.uint8)).astype(np.int64)
    j = np.arange(k, dtype=np.int64)
    p = (j * bits) // 8
    d = (j * bits) % 8
    lo = packed[:, p] >> d[None, :]
    crosses = (d + bits) > 8
    nxt = np.minimum(p + 1, packed.shape[1] - 1)
    hi = np.where(crosses[None, :], packed[:, nxt] << (8 - d)[None, :], 0)
    return (lo | hi) & ((1 << bits) - 1)


def unpack(packed, bits: int, k: int) -> np.ndarray:
    """Signed codes [N, K] from the packed stream."""
    return field_to_code(unpack_fields(packed, bits, k), bits)


# ---------------------------------------------------------------- level function (Sec. 2.2)


def q_curve(t, a, b) -> np.ndarray:
    """q(t) = t [a + t (b + c t)], c = 1 - a - b, in float64 (eq. cubic)."""
    t = np.asarray(t, dtype=np.float64)
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    c = 1.0 - a - b
    return t * (a + t * (b + c * t))


def levels(bits: int, scale: float, a: float, b: float) -> list:
    """Non-negative reconstruction levels of one group (Appendix B).

    W1 returns the pair (-scale, scale); wider widths return s*q(i/M), i=0..M.
    """
    if bits == 1:
        return [-scale, scale]
    m = max_code(bits)
    c = 1.0 - a - b
    out = []
    for i in range(m + 1):
        t = i / m
        out.append(scale * (t * (a + t * (b + t * c))))
    return out


def decode(codes, bits: int, group: int, scale, a_bits, b_bits) -> np.ndarray:
    """Reconstruct w_hat [N, K] in float64 from codes and group metadata.

    B >= 2: w_hat = sign(k) s q(|k|/M) with s widened from FP32 and a, b widened
    exactly from FP16 (eq. cubic).  W1: w_hat = k s.
    """
    codes = np.atleast_2d(np.asarray(codes, dtype=np.int64))
    n, k = codes.shape
    s = np.repeat(np.asarray(scale, dtype=np.float32).astype(np.float64).reshape(n, -1), group, axis=1)
    if bits == 1:
        return codes.astype(np.float64) * s
    a = np.repeat(f16_bits_to_f64(a_bits).reshape(n, -1), group, axis=1)
    b = np.repeat(f16_bits_to_f64(b_bits).reshape(n, -1), group, axis=1)
    m = max_code(bits)
    t = np.abs(codes).astype(np.float64) / m
    return np.sign(codes).astype(np.float64) * s * q_curve(t, a, b)


# ---------------------------------------------------------------- shape domain (Sec. 3.1)


def shape_margin(a, b) -> np.ndarray:
    """m(a, b) = min over t in [0, 1] of q'(t) (eq. shape-domain).

    q'(t) = a + 2 b t + 3 c t^2 with c = 1 - a - b.  Endpoints give a and
    3 - 2a - b; when c > 0 and -3c < b < 0 the interior minimum a - b^2/(3c)
    is included.
    """
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    c = 1.0 - a - b
    ends = np.minimum(a, 3.0 - 2.0 * a - b)
    interior = (c > 0) & (-3.0 * c < b) & (b < 0)
    with np.errstate(divide="ignore", invalid="ignore"):
        inner = np.where(interior, a - b * b / (3.0 * np.where(c > 0, c, 1.0)), np.inf)
    return np.minimum(ends, inner)


def admissible_strict(a, b) -> np.ndarray:
    """Strict monotonicity of the curve: m(a, b) > 0 (eq. monotonicity)."""
    return shape_margin(a, b) > 0


# ---------------------------------------------------------------- storage model (Sec. 2.3, 6.2)


def effective_bits(bits: int, group: int) -> float:
    """B_eff = B + 64/G bits per weight (eq. effective-bits)."""
    return bits + 64.0 / group


def weight_bytes(n: int, k: int, bits: int, group: int) -> float:
    """T_W = N K (B/8 + 8/G) bytes (eq. cubic-weight-bytes)."""
    return n * k * (bits / 8.0 + 8.0 / group)


def bf16_compression(bits: int, group: int) -> float:
    """C = 2 / (B/8 + 8/G) (eq. cubic-bf16-compression)."""
    return 2.0 / (bits / 8.0 + 8.0 / group)
