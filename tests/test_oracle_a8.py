"""Pins for the oracle's Dynamic-A8 semantics (CPU only)."""
from fractions import Fraction

import numpy as np
import pytest

from oracle import a8 as A
from oracle import format as F
from tests.conftest import golden_rows


def test_quantizer_vectors():
    # Sec. 5.4: a row with max |x| = 127 has d_x = 1 exactly; halves round away
    for row in golden_rows("a8_vectors.txt"):
        if row[0] != "row":
            continue
        arrow = row.index("->")
        x = np.array([float(v) for v in row[1:arrow]])[None, :]
        want = np.array([int(v) for v in row[arrow + 1:]])
        x8, d = A.quantize_act(x)
        assert d[0] == np.float32(1.0)
        assert np.array_equal(x8[0], want)


def test_quantizer_half_away_differs_from_rne():
    # 0.5 -> 1, 2.5 -> 3 (nearest-even would give 0 and 2)
    assert A.round_half_away(0.5) == 1 and A.round_half_away(2.5) == 3
    assert A.round_half_away(-2.5) == -3 and A.round_half_away(-0.5) == -1
    assert np.round(2.5) == 2


def test_quantizer_zero_row_uses_epsilon():
    x8, d = A.quantize_act(np.zeros((1, 8)))
    assert np.all(x8 == 0)
    assert d[0] == np.float32(np.float32(1e-10) / np.float32(127.0))


def test_quantizer_correctly_rounded_division():
    # brute force: binary32 division is correctly rounded when the float64
    # quotient is rounded once; compare against exact rational rounding
    rng = np.random.default_rng(0)
    x = rng.standard_normal((20, 257)).astype(np.float32).astype(np.float64)
    x8, d = A.quantize_act(x)
    for m in range(x.shape[0]):
        xbar = max(np.max(np.abs(x[m])), float(np.float32(1e-10)))
        dd = Fraction(float(xbar)) / 127
        d_exact = float(np.float32(float(dd)))  # candidate
        # check d is the binary32 nearest to the exact quotient
        cands = [np.nextafter(np.float32(d_exact), np.float32(-np.inf)), np.float32(d_exact),
                 np.nextafter(np.float32(d_exact), np.float32(np.inf))]
        best = min(cands, key=lambda c: abs(Fraction(float(c)) - dd))
        assert d[m] == best
        for j in range(0, x.shape[1], 17):
            v = Fraction(float(x[m, j])) / Fraction(float(d[m]))
            vf = np.float32(float(v))
            c2 = [np.nextafter(vf, np.float32(-np.inf)), vf, np.nextafter(vf, np.float32(np.inf))]
            vbest = min(c2, key=lambda c: abs(Fraction(float(c)) - v))
            r = np.sign(vbest) * np.floor(abs(float(vbest)) + 0.5)
            assert x8[m, j] == np.clip(r, -127, 127)


def test_quantizer_division_rounding_at_half_max():
    # x = xbar / 2 probes the rounding of x / d_x near 63.5
    x = np.array([[3.0, 1.5, -1.5]])
    x8, d = A.quantize_act(x)
    assert abs(int(x8[0, 1])) in (63, 64)
    assert x8[0, 0] == 127 and x8[0, 2] == -x8[0, 1]


def test_carrier_tie_rounds_to_even():
    # Sec. 4.3 / Appendix A item 7: r = RNE(127 q); 32.5 -> 32
    for row in golden_rows("a8_vectors.txt"):
        if row[0] != "tie":
            continue
        bits, a, b, k, want = int(row[1]), float(row[2]), float(row[3]), int(row[4]), int(row[6])
        a16, b16 = F.f64_to_f16_bits(a), F.f64_to_f16_bits(b)
        assert float(F.f16_bits_to_f64(a16)) == a and float(F.f16_bits_to_f64(b16)) == b
        tab = A.carrier_table(bits, int(a16), int(b16))
        assert tab[k] == want
        # the same value from plain rationals: 127 (a t + b t^2) with c = 0
        t = Fraction(k, 127)
        assert 127 * (Fraction(a) * t + Fraction(b) * t * t) == Fraction(65, 2)


def test_carrier_int_point_is_identity_w8():
    # (a, b) = (1, 0) at W8: r(k) = round(127 k / 127) = k
    tab = A.carrier_table(8, int(F.f64_to_f16_bits(1.0)), int(F.f64_to_f16_bits(0.0)))
    assert tab == list(range(128))


@pytest.mark.parametrize("bits", [1, 2])
def test_w1_w2_carriers_on_grid(bits):
    # W1/W2 levels already lie on the INT8 grid (Sec. 4.3): r in {0, +-127}
    rng = np.random.default_rng(bits)
    a16 = F.f64_to_f16_bits(rng.uniform(0.2, 1.5, (2, 2)))
    b16 = F.f64_to_f16_bits(rng.uniform(-1.0, 0.3, (2, 2)))
    codes = rng.choice(F.valid_codes(bits), size=(2, 64))
    r = A.carriers(codes, bits, 32, a16, b16)
    assert np.array_equal(r, codes * 127)


def test_carrier_exact_vs_float_away_from_ties():
    # brute force: where 127 q is not within 1e-9 of a half-integer, RNE of the
    # float64 value equals the exact rational rounding
    rng = np.random.default_rng(11)
    for _ in range(200):
        bits = int(rng.integers(3, 9))
        a16 = int(F.f64_to_f16_bits(rng.uniform(0.1, 1.5)))
        b16 = int(F.f64_to_f16_bits(rng.uniform(-1.2, 0.4)))
        tab = A.carrier_table(bits, a16, b16)
        a, b = float(F.f16_bits_to_f64(a16)), float(F.f16_bits_to_f64(b16))
        m = F.max_code(bits)
        for i in range(m + 1):
            v = 127 * F.q_curve(i / m, a, b)
            if abs(v - np.floor(v) - 0.5) > 1e-9:
                assert tab[i] == int(np.round(v))


def test_a8_w8_int_point_is_textbook_w8a8():
    # W8 at (1, 0): y = d_x s / 127 * sum x8 k, plain loops
    rng = np.random.default_rng(5)
    n, k, g, m = 3, 64, 32, 2
    codes = rng.integers(-127, 128, (n, k))
    s = rng.uniform(0.01, 0.1, (n, k // g)).astype(np.float32)
    one = np.full((n, k // g), F.f64_to_f16_bits(1.0), np.uint16)
    zero = np.zeros((n, k // g), np.uint16)
    x = rng.standard_normal((m, k)).astype(np.float32).astype(np.float64)
    x8, d = A.quantize_act(x)
    y, p = A.gemm_a8(x8, d, codes, 8, g, s, one, zero)
    for mi in range(m):
        for ni in range(n):
            acc = 0.0
            for gi in range(k // g):
                pg = sum(int(x8[mi, j]) * int(codes[ni, j]) for j in range(gi * g, (gi + 1) * g))
                assert p[mi, ni, gi] == pg
                acc += float(d[mi]) * float(s[ni, gi]) / 127.0 * pg
            assert y[mi, ni] == pytest.approx(acc, rel=1e-13)


def test_int32_bound_is_attained():
    # eq. a8-int32-bound: all +-127 activations and carriers hit G * 127^2
    g = 512
    x8 = np.full((1, g), 127, np.int64)
    r = np.full((1, g), -127, np.int64)
    p = A.group_partials(x8, r, g)
    assert p[0, 0, 0] == -A.int32_bound(g) == -8_258_048
    assert A.int32_bound(512) < 2 ** 31 - 1
