"""Pins for the oracle's real Wigner-D matrices (oracle/wigner.py)."""
import numpy as np
import pytest

from oracle import wigner


@pytest.mark.parametrize("l", [0, 1, 2, 4, 6])
def test_two_constructions_agree(l):
    rng = np.random.default_rng(l)
    for _ in range(3):
        R = wigner.random_rotation(rng)
        np.testing.assert_allclose(wigner.wigner_d_from_sh(l, R), wigner.wigner_d_euler(l, R), atol=1e-11)


@pytest.mark.parametrize("l", [1, 3, 5])
def test_orthogonal_unimodular_homomorphism(l):
    rng = np.random.default_rng(20 + l)
    R1, R2 = wigner.random_rotation(rng), wigner.random_rotation(rng)
    D1, D2 = wigner.wigner_d_from_sh(l, R1), wigner.wigner_d_from_sh(l, R2)
    np.testing.assert_allclose(D1.T @ D1, np.eye(2 * l + 1), atol=1e-12)
    assert abs(np.linalg.det(D1) - 1) < 1e-11
    np.testing.assert_allclose(wigner.wigner_d_from_sh(l, R1 @ R2), D1 @ D2, atol=1e-11)


def test_degree_one_is_permuted_rotation():
    rng = np.random.default_rng(7)
    R = wigner.random_rotation(rng)
    P = np.array([[0, 1, 0], [0, 0, 1], [1, 0, 0.0]])   # (x, y, z) -> (y, z, x)
    np.testing.assert_allclose(wigner.wigner_d_from_sh(1, R), P @ R @ P.T, atol=1e-12)


def test_random_rotation_is_rotation():
    rng = np.random.default_rng(8)
    R = wigner.random_rotation(rng)
    np.testing.assert_allclose(R @ R.T, np.eye(3), atol=1e-14)
    assert abs(np.linalg.det(R) - 1) < 1e-13
