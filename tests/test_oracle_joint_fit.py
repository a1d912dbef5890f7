"""Pins for the oracle's carrier-aware joint fitter (Sec. 4.3; CPU only)."""
import numpy as np
import pytest

from oracle import a8 as A8
from oracle import fit as FIT
from oracle import format as F
from tests._cases import near_tie_shapes
from workloads import small_weight


def test_c_carriers_equal_the_exact_table():
    # the joint scorer's integer carriers against the Fraction-based table
    # (eq. carrier, RNE of the exact value), on the coarse grid and on shapes
    # searched to sit next to a carrier tie
    ca, cb = FIT.coarse_candidates()
    for bits in range(2, 9):
        shapes = list(zip(ca, cb))
        if bits >= 3:
            shapes += [(float(F.f16_bits_to_f64(a)), float(F.f16_bits_to_f64(b)))
                       for a, b in near_tie_shapes(bits, count=16)]
        for a, b in shapes:
            ab, bb = F.f64_to_f16_bits(a), F.f64_to_f16_bits(b)
            want = A8.carrier_table(bits, int(ab), int(bb))
            assert list(FIT.carriers_c(bits, a, b)) == want, (bits, a, b)


def test_joint_w1_w2_equal_the_continuous_fit():
    # W1 and W2 levels lie on the carrier grid, so L_C = L_A8 and the joint
    # objective is twice the continuous one: same representation
    w = small_weight(21, 8, 256, "laplace")
    for bits in (1, 2):
        rj = FIT.fit_joint(w, bits, 128)
        rc = FIT.fit(w, bits, 128)
        assert np.array_equal(rj.codes, rc.codes)
        assert np.array_equal(rj.scale, rc.scale)
        assert np.allclose(rj.loss_c, rj.loss_a8)


def test_joint_codes_are_joint_argmin():
    # eq. carrier-aware-assignment: under the stored (s, a, b) every code's
    # magnitude minimises (u - s q)^2 + (u - s r / 127)^2, ties to the smaller
    w = small_weight(22, 4, 64, "laplace")
    for bits in (3, 4, 5, 6):
        r = FIT.fit_joint(w, bits, 16)
        for row in range(4):
            for gi in range(4):
                s = float(r.scale[row, gi])
                ab, bb = int(r.a_bits[row, gi]), int(r.b_bits[row, gi])
                lv = np.array(F.levels(bits, s, float(F.f16_bits_to_f64(ab)), float(F.f16_bits_to_f64(bb))))
                car = np.array(A8.carrier_table(bits, ab, bb), np.float64)
                for j in range(gi * 16, gi * 16 + 16):
                    u = abs(float(w[row, j]))
                    cost = (u - lv) ** 2 + (u - s * car / 127.0) ** 2
                    assert abs(int(r.codes[row, j])) == int(np.argmin(cost))


def test_joint_losses_are_those_of_the_representation():
    # the fitter's reported L_C and L_A8 equal an independent evaluation of
    # the stored representation (decode + exact carrier table)
    w = small_weight(23, 6, 512, "normal")
    for bits in (3, 4, 8):
        r = FIT.fit_joint(w, bits, 128)
        lc, la = FIT.joint_loss(w, r.codes, bits, 128, r.scale, r.a_bits, r.b_bits)
        assert np.allclose(lc, r.loss_c, rtol=1e-9, atol=1e-18)
        assert np.allclose(la, r.loss_a8, rtol=1e-9, atol=1e-18)


@pytest.mark.parametrize("law", ["laplace", "normal"])
def test_joint_fit_improves_the_a8_representation(law):
    # the joint objective is what the joint fit minimises: on aggregate it
    # is no worse than the continuous fit's representation scored the same
    # way, and the A8 error (sqrt(L_A8 / sum w^2)) improves at W3..W6
    w = small_weight(24, 16, 1024, law)
    for bits in (3, 4, 5, 6):
        rj = FIT.fit_joint(w, bits, 128)
        rc = FIT.fit(w, bits, 128)
        lc_c, la_c = FIT.joint_loss(w, rc.codes, bits, 128, rc.scale, rc.a_bits, rc.b_bits)
        assert (rj.loss_c + rj.loss_a8).sum() <= (lc_c + la_c).sum()
        assert rj.loss_a8.sum() < la_c.sum()
        # eq. carrier-aware-nrmse
        ww = np.sum(w.astype(np.float64) ** 2)
        assert rj.nrmse_joint(w) == pytest.approx(np.sqrt((rj.loss_c.sum() + rj.loss_a8.sum()) / (2 * ww)))


def test_joint_brute_force_tiny_groups():
    # G = 8, W3: a dense scan of s over every coarse candidate, each weight
    # taking its joint argmin, cannot beat the fitter by more than a small
    # margin
    w = small_weight(25, 6, 8, "laplace")
    bits = 3
    r = FIT.fit_joint(w, bits, 8)
    ca, cb = FIT.coarse_candidates()
    for row in range(6):
        u = np.abs(w[row].astype(np.float64))
        best = np.inf
        for a, b in zip(ca, cb):
            z = np.array(F.levels(bits, 1.0, a, b))
            zt = np.array(A8.carrier_table(bits, int(F.f64_to_f16_bits(a)), int(F.f64_to_f16_bits(b))),
                          np.float64) / 127.0
            for s in np.linspace(0.3, 1.3, 401) * u.max():
                cost = (u[:, None] - s * z[None, :]) ** 2 + (u[:, None] - s * zt[None, :]) ** 2
                best = min(best, float(np.sum(np.min(cost, axis=1))))
        assert r.loss_c[row, 0] + r.loss_a8[row, 0] <= best * 1.02 + 1e-18
