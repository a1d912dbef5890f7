"""Pins for the oracle's storage format and level function (CPU only).

Each check compares the oracle with something the paper or plain mathematics
fixes independently of the oracle's own code: hand-worked byte vectors, the
uniform-integer special case, exact endpoints, the reference decode of
Appendix B written out here as scalar Python, a brute-force minimum of q'
and the printed storage tables.
"""
import itertools

import numpy as np
import pytest

from oracle import format as F
from tests.conftest import golden_rows


def _hex(bs):
    return " ".join(f"{b:02x}" for b in bs)


@pytest.mark.parametrize("row", [r for r in golden_rows("pack_vectors.txt") if r[0] != "reserved"])
def test_worked_pack_vectors(row):
    # Sec. 2.1 / eq. gpu-packed-extraction, worked by hand
    arrow = row.index("->")
    bits = int(row[0])
    codes = np.array([int(c) for c in row[1:arrow]])
    want = " ".join(row[arrow + 1:])
    packed = F.pack(codes[None, :], bits)[0]
    assert _hex(packed) == want
    assert np.array_equal(F.unpack(packed[None, :], bits, len(codes))[0], codes)


@pytest.mark.parametrize("row", [r for r in golden_rows("pack_vectors.txt") if r[0] == "reserved"])
def test_reserved_pattern_decodes_to_zero(row):
    # Sec. 2.1 and Appendix A item 2
    bits, k = int(row[1]), int(row[2])
    packed = np.array([int(h, 16) for h in row[3:]], dtype=np.uint8)[None, :]
    assert np.all(F.unpack(packed, bits, k) == 0)
    assert np.all(F.unpack_fields(packed, bits, k) == (1 << (bits - 1)))


@pytest.mark.parametrize("bits", range(1, 9))
def test_roundtrip_all_widths(bits):
    rng = np.random.default_rng(bits)
    for k in (8, 24, 64, 128, 136):
        if (k * bits) % 8:
            continue
        codes = rng.choice(F.valid_codes(bits), size=(5, k))
        packed = F.pack(codes, bits)
        assert packed.shape == (5, k * bits // 8)
        assert np.array_equal(F.unpack(packed, bits, k), codes)


def test_pack_matches_bit_definition_by_brute_force():
    # stream bit p is bit (p mod 8) of byte p // 8; field j occupies [jB, jB+B)
    rng = np.random.default_rng(7)
    for bits in range(1, 9):
        k = 16
        codes = rng.choice(F.valid_codes(bits), size=(1, k))
        packed = F.pack(codes, bits)[0]
        for j in range(k):
            kj = int(codes[0, j])
            field = (1 if kj > 0 else 0) if bits == 1 else kj % (1 << bits)
            for b in range(bits):
                p = j * bits + b
                assert ((packed[p // 8] >> (p % 8)) & 1) == ((field >> b) & 1)


def test_reserved_never_emitted_and_rejected():
    for bits in range(2, 9):
        with pytest.raises(ValueError):
            F.pack(np.array([[-(1 << (bits - 1))]]), bits)
    with pytest.raises(ValueError):
        F.pack(np.array([[0]]), 1)


def _appendix_b_levels(bits, scale, a, b):
    # Appendix B reference decode written out as scalar Python
    if bits == 1:
        return (-scale, scale)
    maximum = (1 << (bits - 1)) - 1
    c = 1.0 - a - b
    out = []
    for index in range(maximum + 1):
        t = index / maximum
        out.append(scale * (t * (a + t * (b + t * c))))
    return out


@pytest.mark.parametrize("bits", range(1, 9))
def test_decode_matches_appendix_b(bits):
    rng = np.random.default_rng(100 + bits)
    g = 32
    n, k = 3, 64
    codes = rng.choice(F.valid_codes(bits), size=(n, k))
    scale = rng.uniform(0.01, 2.0, (n, k // g)).astype(np.float32)
    a16 = F.f64_to_f16_bits(rng.uniform(0.3, 1.2, (n, k // g)))
    b16 = F.f64_to_f16_bits(rng.uniform(-0.5, 0.1, (n, k // g)))
    w = F.decode(codes, bits, g, scale, a16, b16)
    for r in range(n):
        for j in range(k):
            gi = j // g
            s = float(scale[r, gi])
            a = float(F.f16_bits_to_f64(a16[r, gi]))
            b = float(F.f16_bits_to_f64(b16[r, gi]))
            lv = _appendix_b_levels(bits, s, a, b)
            kj = int(codes[r, j])
            if bits == 1:
                want = lv[1] if kj > 0 else lv[0]
            else:
                want = (1 if kj > 0 else -1 if kj < 0 else 0) * lv[abs(kj)]
            assert w[r, j] == pytest.approx(want, rel=1e-15, abs=1e-300)


@pytest.mark.parametrize("bits", range(2, 9))
def test_int_special_case(bits):
    # eq. int-special-case: (a, b) = (1, 0) gives w_hat = s k / M exactly
    m = F.max_code(bits)
    codes = F.valid_codes(bits)[None, :]
    k = codes.shape[1]
    scale = np.array([[0.75]], np.float32)
    one = F.f64_to_f16_bits([[1.0]])
    zero = F.f64_to_f16_bits([[0.0]])
    w = F.decode(codes, bits, k, scale, one, zero)
    assert np.allclose(w, 0.75 * codes / m, rtol=1e-15, atol=0)


@pytest.mark.parametrize("bits", range(2, 9))
def test_endpoints_exact_and_levels_monotone(bits):
    # Sec. 2.2: q(0) = 0 and q(1) = 1 for any (a, b); strictly increasing levels
    # whenever m(a, b) > 0 (eq. monotonicity)
    m = F.max_code(bits)
    rng = np.random.default_rng(bits)
    for _ in range(50):
        a = float(F.f16_bits_to_f64(F.f64_to_f16_bits(rng.uniform(0.05, 2.0))))
        b = float(F.f16_bits_to_f64(F.f64_to_f16_bits(rng.uniform(-1.5, 1.0))))
        lv = np.array(F.levels(bits, 1.0, a, b))
        assert lv[0] == 0.0
        assert lv[-1] == pytest.approx(1.0, abs=1e-15)
        if F.admissible_strict(a, b):
            assert np.all(np.diff(lv) > 0)
        codes = np.array([[m, -m, 0]])
        w = F.decode(codes, bits, 3, np.array([[0.5]], np.float32),
                     F.f64_to_f16_bits([[a]]), F.f64_to_f16_bits([[b]]))
        assert w[0, 0] == pytest.approx(0.5, abs=1e-15) and w[0, 1] == pytest.approx(-0.5, abs=1e-15)
        assert w[0, 2] == 0.0


def test_shape_margin_matches_dense_grid_minimum():
    # eq. shape-domain against brute force min of q'(t) on a fine grid
    t = np.linspace(0.0, 1.0, 20001)
    rng = np.random.default_rng(3)
    for _ in range(400):
        a = rng.uniform(-0.5, 3.5)
        b = rng.uniform(-4.0, 3.0)
        c = 1 - a - b
        brute = np.min(a + 2 * b * t + 3 * c * t * t)
        assert F.shape_margin(a, b) == pytest.approx(brute, abs=1e-6)


def test_shape_margin_known_points():
    assert F.shape_margin(1.0, 0.0) == 1.0          # q(t) = t
    assert F.shape_margin(0.8, -0.4) > 0            # Sec. 2.2 figure members
    assert F.shape_margin(0.5, -0.3) > 0
    assert F.shape_margin(0.0, 0.0) == 0.0          # q(t) = t^3: closure only
    assert not F.admissible_strict(0.0, 0.0)
    assert F.shape_margin(2.0, 0.0) < 0             # q'(1) = 3 - 4 < 0


def test_storage_tables(golden):
    # Sec. 6.2 storage table and Sec. 2.3 effective widths
    for row in golden("storage.txt"):
        if row[0] == "G":
            g, extra = int(row[1]), float(row[2])
            for bits in range(1, 9):
                assert F.effective_bits(bits, g) == pytest.approx(bits + extra)
            continue
        bits = int(row[0])
        assert F.weight_bytes(1, 1, bits, 256) == pytest.approx(float(row[1]))
        assert F.bf16_compression(bits, 256) == pytest.approx(float(row[2]), abs=0.006)
        assert F.weight_bytes(1, 1, bits, 512) == pytest.approx(float(row[3]))
        assert F.bf16_compression(bits, 512) == pytest.approx(float(row[4]), abs=0.006)


def test_weight_bytes_w4_g128_4096():
    # 4096 x 4096 W4 G128: 8 MiB of codes + 1 MiB of metadata
    assert F.weight_bytes(4096, 4096, 4, 128) == 9_437_184


def test_w1_decode_is_plus_minus_scale():
    codes = np.array([[1, -1, 1, -1]])
    w = F.decode(codes, 1, 4, np.array([[0.25]], np.float32), np.zeros((1, 1), np.uint16),
                 np.zeros((1, 1), np.uint16))
    assert np.array_equal(w, [[0.25, -0.25, 0.25, -0.25]])


def test_field_code_exhaustive():
    for bits in range(2, 9):
        half = 1 << (bits - 1)
        for u, in itertools.product(range(1 << bits)):
            k = int(F.field_to_code(u, bits))
            if u == half:
                assert k == 0
            elif u < half:
                assert k == u
            else:
                assert k == u - (1 << bits)
