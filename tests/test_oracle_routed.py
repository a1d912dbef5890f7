"""Pins for the oracle's routed (mixture-of-experts) product (CPU only)."""
import numpy as np
import pytest

from oracle import format as F
from oracle import routed as RT
from workloads import bf16_bits_to_f32, route_map, small_act


def _bank(seed, experts, n, k, bits, g, int_point=False):
    rng = np.random.default_rng(seed)
    mm = F.max_code(bits)
    codes = rng.integers(-mm, mm + 1, (experts * n, k))
    s = rng.uniform(0.01, 0.05, (experts * n, k // g)).astype(np.float32)
    if int_point:
        a = np.full(s.shape, F.f64_to_f16_bits(1.0), np.uint16)
        b = np.zeros(s.shape, np.uint16)
    else:
        a = np.full(s.shape, F.f64_to_f16_bits(0.7932), np.uint16)
        b = np.full(s.shape, F.f64_to_f16_bits(-0.3847), np.uint16)
    return codes, s, a, b


def test_routed_int_point_is_groupwise_int_per_route():
    # at (a, b) = (1, 0) every route is sum_j x_{t,j} s_{e,g} k_{e,j} / M,
    # evaluated here with explicit loops over the routes and K
    bits, g, n, k, experts = 4, 32, 3, 64, 3
    mm = F.max_code(bits)
    codes, s, a, b = _bank(5, experts, n, k, bits, g, int_point=True)
    x = bf16_bits_to_f32(small_act(6, 4, k)).astype(np.float64)
    tok = np.array([2, 0, 3, 2, 1], np.int32)
    exp = np.array([1, 2, 0, 0, 2], np.int32)
    y = RT.routed_model_dtype(x, tok, exp, codes, bits, g, s, a, b, experts)
    for r in range(len(tok)):
        for j in range(n):
            row = exp[r] * n + j
            acc = 0.0
            for c in range(k):
                acc += x[tok[r], c] * float(s[row, c // g]) * codes[row, c] / mm
            assert y[r, j] == pytest.approx(acc, rel=1e-12, abs=1e-15)


def test_routed_cubic_naive_loops():
    # a cubic shape: levels from the explicit curve s sign(k) q(|k|/M), q(t) = t (a + b t + c t^2)
    bits, g, n, k, experts = 3, 32, 2, 64, 2
    mm = F.max_code(bits)
    codes, s, a, b = _bank(7, experts, n, k, bits, g)
    av, bv = 0.7932, -0.3847
    aa = F.f16_bits_to_f64(np.array([F.f64_to_f16_bits(av)]))[0]
    bb = F.f16_bits_to_f64(np.array([F.f64_to_f16_bits(bv)]))[0]
    cc = 1.0 - aa - bb
    x = bf16_bits_to_f32(small_act(8, 3, k)).astype(np.float64)
    tok = np.array([0, 2, 1], np.int32)
    exp = np.array([1, 0, 1], np.int32)
    y = RT.routed_model_dtype(x, tok, exp, codes, bits, g, s, a, b, experts)
    for r in range(3):
        for j in range(n):
            row = exp[r] * n + j
            acc = 0.0
            for c in range(k):
                kk = int(codes[row, c])
                t = abs(kk) / mm
                q = t * (aa + bb * t + cc * t * t)
                acc += x[tok[r], c] * float(s[row, c // g]) * np.sign(kk) * q
            assert y[r, j] == pytest.approx(acc, rel=1e-12, abs=1e-15)


def test_routed_route_order_permutes_rows_only():
    bits, g, n, k, experts = 4, 32, 4, 96, 4
    codes, s, a, b = _bank(9, experts, n, k, bits, g)
    x = bf16_bits_to_f32(small_act(10, 6, k)).astype(np.float64)
    tok, exp = route_map(11, 6, experts, 2)
    y = RT.routed_model_dtype(x, tok, exp, codes, bits, g, s, a, b, experts)
    perm = np.random.default_rng(12).permutation(len(tok))
    y2 = RT.routed_model_dtype(x, tok[perm], exp[perm], codes, bits, g, s, a, b, experts)
    assert np.array_equal(y2, y[perm])


def test_routed_invalid_routes_have_no_row():
    bits, g, n, k, experts = 4, 32, 2, 64, 2
    codes, s, a, b = _bank(13, experts, n, k, bits, g)
    x = bf16_bits_to_f32(small_act(14, 2, k)).astype(np.float64)
    y = RT.routed_model_dtype(x, [0, 2, 1, -1], [1, 0, 2, 0], codes, bits, g, s, a, b, experts)
    assert np.all(np.isfinite(y[0])) and np.all(np.isnan(y[1:]))


def test_route_map_shape_and_distinct_experts():
    tok, exp = route_map(15, 33, 8, 2)
    assert len(tok) == 66 and tok.dtype == np.int32 and exp.dtype == np.int32
    for t in range(33):
        e = exp[tok == t]
        assert len(e) == 2 and e[0] != e[1] and np.all((0 <= e) & (e < 8))
