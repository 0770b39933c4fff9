"""Pins for the oracle's real spherical harmonics (oracle/sh.py).

Independent references: textbook closed forms for l <= 2, the addition
theorem, quadrature orthogonality on the sphere, scipy's complex harmonics
(through the basis change of oracle.cg), and finite differences."""
import numpy as np
import pytest
from scipy.special import sph_harm_y

from oracle import cg, sh


def _unit(rng, n):
    u = rng.normal(size=(n, 3))
    return u / np.linalg.norm(u, axis=1, keepdims=True)


def test_low_degree_closed_forms():
    rng = np.random.default_rng(0)
    u = _unit(rng, 50)
    x, y, z = u.T
    Y = sh.solid_harmonics(2, u)
    s3, s15, s5 = np.sqrt(3), np.sqrt(15), np.sqrt(5)
    ref = np.stack([np.ones_like(x),
                    s3 * y, s3 * z, s3 * x,
                    s15 * x * y, s15 * y * z, s5 / 2 * (3 * z * z - 1), s15 * x * z,
                    s15 / 2 * (x * x - y * y)], 1)
    np.testing.assert_allclose(Y, ref, atol=1e-13)


@pytest.mark.parametrize("L", [0, 1, 3, 6])
def test_addition_theorem(L):
    rng = np.random.default_rng(L)
    Y = sh.spherical_harmonics(L, rng.normal(size=(200, 3)) * 3.0)
    for l in range(L + 1):
        s = np.sum(Y[:, l * l:(l + 1) ** 2] ** 2, axis=1)
        np.testing.assert_allclose(s, 2 * l + 1, rtol=1e-12)


def test_quadrature_orthogonality():
    L = 6
    nt, nphi = 2 * L + 2, 2 * L + 3
    t, wt = np.polynomial.legendre.leggauss(nt)          # z = cos(theta)
    phi = 2 * np.pi * np.arange(nphi) / nphi
    T, P = np.meshgrid(t, phi, indexing="ij")
    st = np.sqrt(1 - T * T)
    u = np.stack([st * np.cos(P), st * np.sin(P), T], -1).reshape(-1, 3)
    w = (wt[:, None] * np.full(nphi, 2 * np.pi / nphi)[None, :]).reshape(-1)
    Y = sh.solid_harmonics(L, u)
    gram = (Y * w[:, None]).T @ Y
    np.testing.assert_allclose(gram, 4 * np.pi * np.eye((L + 1) ** 2), atol=1e-11)


@pytest.mark.parametrize("L", [1, 2, 4, 6])
def test_matches_scipy_complex_harmonics(L):
    rng = np.random.default_rng(10 + L)
    u = _unit(rng, 40)
    theta = np.arccos(u[:, 2])
    phi = np.arctan2(u[:, 1], u[:, 0])
    Y = sh.solid_harmonics(L, u)
    for l in range(L + 1):
        ms = np.arange(-l, l + 1)
        Yc = np.stack([sph_harm_y(l, m, theta, phi) for m in ms], 1)   # orthonormal, CS phase
        Yr = np.sqrt(4 * np.pi) * Yc @ cg.complex_to_real(l).T
        np.testing.assert_allclose(Yr.imag, 0, atol=1e-12)
        np.testing.assert_allclose(Y[:, l * l:(l + 1) ** 2], Yr.real, atol=1e-11)


def test_solid_harmonics_are_homogeneous():
    rng = np.random.default_rng(3)
    r = rng.normal(size=(20, 3))
    L = 5
    ls = np.concatenate([np.full(2 * l + 1, l) for l in range(L + 1)])
    np.testing.assert_allclose(sh.solid_harmonics(L, 2.5 * r), 2.5 ** ls * sh.solid_harmonics(L, r),
                               rtol=1e-11, atol=1e-11)


@pytest.mark.parametrize("L", [2, 6])
def test_gradient_finite_difference(L):
    rng = np.random.default_rng(4)
    r = rng.normal(size=(10, 3))
    g = sh.solid_harmonics_grad(L, r)
    h = 1e-6
    for a in range(3):
        dr = np.zeros(3)
        dr[a] = h
        fd = (sh.solid_harmonics(L, r + dr) - sh.solid_harmonics(L, r - dr)) / (2 * h)
        np.testing.assert_allclose(g[..., a], fd, rtol=1e-6, atol=1e-6)


@pytest.mark.parametrize("L", [1, 4, 6])
def test_direction_jacobian_finite_difference(L):
    rng = np.random.default_rng(5)
    v = rng.normal(size=(10, 3)) * 2.0
    J = sh.spherical_harmonics_jacobian(L, v)
    h = 1e-6
    for a in range(3):
        dv = np.zeros(3)
        dv[a] = h
        fd = (sh.spherical_harmonics(L, v + dv) - sh.spherical_harmonics(L, v - dv)) / (2 * h)
        np.testing.assert_allclose(J[..., a], fd, rtol=1e-6, atol=1e-6)
    # Y depends on the direction only: J v = 0
    np.testing.assert_allclose(np.einsum("ekx,ex->ek", J, v), 0, atol=1e-10)
