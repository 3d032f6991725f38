"""Pins of the oracle's radial basis, envelope, SiLU family and Legendre
polynomials against closed forms, integrals and library routines."""
import numpy as np
import pytest
from scipy import integrate, special

from oracle.basis import bessel_basis, envelope, legendre, silu, silu_d1, silu_d2, silu_family


def test_envelope_vanishes_to_second_order_at_cutoff():
    u, du, d2u = envelope(np.array([0.0, 1.0, 1.5]))
    assert u[0] == 1.0 and du[0] == 0.0 and d2u[0] == 0.0
    # polynomial identities at x = 1: 1-28+48-21, -168+336-168, -840+2016-1176
    assert u[1] == 0.0 and du[1] == 0.0 and d2u[1] == 0.0
    assert u[2] == 0.0 and du[2] == 0.0 and d2u[2] == 0.0


def test_envelope_derivatives_match_finite_differences():
    x = np.linspace(0.05, 0.97, 37)
    h = 1e-6
    u, du, d2u = envelope(x)
    up, dup, _ = envelope(x + h)
    um, dum, _ = envelope(x - h)
    np.testing.assert_allclose((up - um) / (2 * h), du, rtol=1e-7, atol=1e-9)
    np.testing.assert_allclose((dup - dum) / (2 * h), d2u, rtol=1e-6, atol=1e-8)


@pytest.mark.parametrize("rc,nb", [(4.0, 8), (6.0, 16)])
def test_unenveloped_bessel_functions_are_orthonormal(rc, nb):
    # integral_0^rc (2/rc) sin(m pi r/rc) sin(n pi r/rc) / r^2 * r^2 dr = delta_mn
    def b(n, r):
        return np.sqrt(2.0 / rc) * np.sin(n * np.pi * r / rc) / r
    for m in (1, 2, nb):
        for n in (1, 3, nb):
            val, _ = integrate.quad(lambda r: b(m, r) * b(n, r) * r * r, 0.0, rc, limit=200)
            assert abs(val - (1.0 if m == n else 0.0)) < 1e-10


def test_basis_is_bessel_times_envelope_and_limits():
    rc, nb = 5.0, 16
    r = np.array([1e-4, 0.7, 2.5, 4.999])
    B, dB, d2B = bessel_basis(r, rc, nb)
    n = np.arange(1, nb + 1)
    u, _, _ = envelope(r / rc)
    ref = np.sqrt(2.0 / rc) * np.sin(np.outer(r, n) * np.pi / rc) / r[:, None] * u[:, None]
    np.testing.assert_allclose(B, ref, rtol=1e-12)
    # r -> 0+: sin(k r)/r -> k, envelope -> 1
    np.testing.assert_allclose(B[0], np.sqrt(2.0 / rc) * n * np.pi / rc, rtol=1e-6)
    # near the cutoff all three vanish (cubic order in rc - r)
    assert np.abs(B[-1]).max() < 1e-7 and np.abs(dB[-1]).max() < 1e-4


def test_basis_derivatives_match_finite_differences():
    rc, nb = 6.0, 16
    r = np.linspace(0.3, 5.9, 57)
    h = 1e-6
    B, dB, d2B = bessel_basis(r, rc, nb)
    Bp, dBp, _ = bessel_basis(r + h, rc, nb)
    Bm, dBm, _ = bessel_basis(r - h, rc, nb)
    np.testing.assert_allclose((Bp - Bm) / (2 * h), dB, rtol=1e-6, atol=1e-8)
    np.testing.assert_allclose((dBp - dBm) / (2 * h), d2B, rtol=1e-5, atol=1e-7)


def test_silu_family_closed_forms_and_finite_differences():
    a = np.linspace(-12, 12, 241)
    h = 1e-6
    np.testing.assert_allclose(silu(a), a / (1.0 + np.exp(-a)), rtol=1e-14, atol=1e-300)
    np.testing.assert_allclose((silu(a + h) - silu(a - h)) / (2 * h), silu_d1(a), rtol=1e-7, atol=1e-9)
    np.testing.assert_allclose((silu_d1(a + h) - silu_d1(a - h)) / (2 * h), silu_d2(a), rtol=1e-6, atol=1e-8)
    assert silu_d1(0.0) == 0.5 and silu_d2(0.0) == 0.5
    s0, s1, s2 = silu_family(np.tile(a, (5000, 1)))        # threaded path
    np.testing.assert_allclose(s0[17], silu(a), rtol=1e-14, atol=1e-300)
    np.testing.assert_allclose(s1[4999], silu_d1(a), rtol=1e-14, atol=1e-15)
    np.testing.assert_allclose(s2[0], silu_d2(a), rtol=1e-14, atol=1e-15)


def test_legendre_against_library_and_identities():
    x = np.linspace(-1, 1, 101)
    P, dP = legendre(x, 5)
    for l in range(5):
        np.testing.assert_allclose(P[:, l], special.eval_legendre(l, x), rtol=1e-13, atol=1e-14)
        assert P[-1, l] == pytest.approx(1.0) and P[0, l] == pytest.approx((-1.0) ** l)
        h = 1e-6
        xi = np.linspace(-0.9, 0.9, 19)
        Pp, _ = legendre(xi + h, 5)
        Pm, _ = legendre(xi - h, 5)
        _, dPi = legendre(xi, 5)
        np.testing.assert_allclose((Pp[:, l] - Pm[:, l]) / (2 * h), dPi[:, l], rtol=1e-6, atol=1e-8)
