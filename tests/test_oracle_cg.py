"""Pins for the oracle's CG coefficients and CG tensor (oracle/cg.py,
oracle/cg_tensor.py).

Independent references: sympy's exact CG, the two orthogonality relations,
selection rules, the worked l1 = l2 = 1 case of Sec. 3.1 (Fig. 1: outputs of
degree 0, 1, 2 are the dot product, the cross product and the symmetric
traceless part), closed forms for ||M||_F and its mode Gram diagonals, and
exact equivariance under Wigner-D matrices built from the harmonics."""
import itertools

import numpy as np
import pytest
from sympy import S
from sympy.physics.wigner import clebsch_gordan

from oracle import cg, cg_tensor, wigner


@pytest.mark.parametrize("l1,l2,l3", [(1, 1, 2), (2, 1, 3), (2, 2, 2), (3, 2, 4), (4, 3, 2), (6, 6, 6)])
def test_complex_cg_matches_sympy(l1, l2, l3):
    for m1 in range(-l1, l1 + 1):
        for m2 in range(-l2, l2 + 1):
            m3 = m1 + m2
            if abs(m3) > l3:
                continue
            ref = float(clebsch_gordan(S(l1), S(l2), S(l3), S(m1), S(m2), S(m3)))
            assert abs(cg.cg_complex(l1, m1, l2, m2, l3, m3) - ref) < 1e-13


def test_orthogonality_relations():
    L = 4
    for l1, l2 in itertools.product(range(L + 1), repeat=2):
        blocks = {l3: cg.cg_complex_block(l1, l2, l3) for l3 in range(abs(l1 - l2), l1 + l2 + 1)}
        # sum_{m1 m2} C^{l3 m3} C^{l3' m3'} = delta
        for l3, C3 in blocks.items():
            for l3p, C3p in blocks.items():
                G = np.einsum("aij,bij->ab", C3, C3p)
                ref = np.eye(2 * l3 + 1) if l3 == l3p else 0
                np.testing.assert_allclose(G, ref, atol=1e-13)
            # sum_{m2 m3} C C = (2l3+1)/(2l1+1) delta_{m1 m1'}
            G1 = np.einsum("aij,akj->ik", C3, C3)
            np.testing.assert_allclose(G1, (2 * l3 + 1) / (2 * l1 + 1) * np.eye(2 * l1 + 1), atol=1e-13)


def test_selection_rules_and_identity():
    assert cg.cg_complex(2, 1, 1, 1, 3, 1) == 0.0           # m3 != m1 + m2
    assert cg.cg_complex(3, 0, 1, 0, 1, 0) == 0.0           # outside triangle
    for l in range(5):
        Cb = cg.cg_complex_block(0, l, l)[:, 0, :]
        np.testing.assert_allclose(Cb, np.eye(2 * l + 1), atol=1e-15)


@pytest.mark.parametrize("l1,l2,l3", [(1, 1, 1), (2, 1, 2), (3, 3, 3), (2, 2, 3), (4, 2, 3)])
def test_real_blocks_are_real_and_orthonormal(l1, l2, l3):
    Cr = cg.cg_real(l1, l2, l3)
    G = np.einsum("aij,bij->ab", Cr, Cr)
    np.testing.assert_allclose(G, np.eye(2 * l3 + 1), atol=1e-13)


def _cart(v):
    """degree-1 real components are ordered (y, z, x)."""
    return np.array([v[2], v[0], v[1]])


def test_figure1_case_l1_l2_equal_1():
    rng = np.random.default_rng(0)
    a, b = rng.normal(size=3), rng.normal(size=3)
    ya = np.array([a[1], a[2], a[0]])
    yb = np.array([b[1], b[2], b[0]])
    out0 = np.einsum("kij,i,j->k", cg.cg_real(1, 1, 0), ya, yb)
    out1 = np.einsum("kij,i,j->k", cg.cg_real(1, 1, 1), ya, yb)
    out2 = np.einsum("kij,i,j->k", cg.cg_real(1, 1, 2), ya, yb)
    # degree 0: proportional to the dot product with the orthonormal factor 1/sqrt(3)
    assert abs(abs(out0[0]) - abs(a @ b) / np.sqrt(3)) < 1e-13
    # degree 1: proportional to the cross product, factor 1/sqrt(2)
    cr = np.cross(a, b)
    c1 = _cart(out1)
    np.testing.assert_allclose(np.abs(c1), np.abs(cr) / np.sqrt(2), atol=1e-13)
    assert abs(abs(c1 @ cr) - (cr @ cr) / np.sqrt(2)) < 1e-12
    # degree 2: depends only on the symmetric traceless part of a b^T
    Sab = 0.5 * (np.outer(a, b) + np.outer(b, a))
    Sab -= np.trace(Sab) / 3 * np.eye(3)
    # same output for a pair with the same symmetric traceless part: swap a, b
    out2s = np.einsum("kij,i,j->k", cg.cg_real(1, 1, 2), yb, ya)
    np.testing.assert_allclose(out2, out2s, atol=1e-13)
    assert abs(np.linalg.norm(out2) - np.linalg.norm(Sab)) < 1e-12
    # and antisymmetric/trace parts do not enter: a b^T - b a^T gives zero
    np.testing.assert_allclose(out0, np.einsum("kij,i,j->k", cg.cg_real(1, 1, 0), yb, ya), atol=1e-13)


@pytest.mark.parametrize("L,frob2,npaths", [(1, 11, 5), (2, 51, 15), (3, 156, 34), (4, 375, 65),
                                            (5, 771, 111), (6, 1421, 175)])
def test_tensor_norm_and_path_count(L, frob2, npaths):
    M = cg_tensor.cg_tensor(L)
    assert len(cg_tensor.paths(L)) == npaths
    assert abs(np.sum(M * M) - frob2) < 1e-9
    assert frob2 == sum(2 * l3 + 1 for _, _, l3 in cg_tensor.paths(L))


@pytest.mark.parametrize("L", [2, 3, 5])
def test_mode_gram_diagonals(L):
    M = cg_tensor.cg_tensor(L)
    P = cg_tensor.paths(L)
    g_out = np.einsum("kij,kij->k", M, M)
    g_x = np.einsum("kij,kij->i", M, M)
    g_y = np.einsum("kij,kij->j", M, M)
    for l in range(L + 1):
        sl = slice(l * l, (l + 1) ** 2)
        np.testing.assert_allclose(g_out[sl], sum(1 for p in P if p[2] == l), atol=1e-11)
        np.testing.assert_allclose(g_x[sl], sum((2 * p[2] + 1) / (2 * l + 1) for p in P if p[0] == l),
                                   atol=1e-11)
        np.testing.assert_allclose(g_y[sl], sum((2 * p[2] + 1) / (2 * l + 1) for p in P if p[1] == l),
                                   atol=1e-11)


@pytest.mark.parametrize("L", [2, 4, 6])
def test_dense_product_exactly_equivariant(L):
    rng = np.random.default_rng(L)
    M = cg_tensor.cg_tensor(L)
    d = (L + 1) ** 2
    for _ in range(3):
        R = wigner.random_rotation(rng)
        Drot = wigner.wigner_d_full(L, R)
        x, y = rng.normal(size=(2, d))
        lhs = cg_tensor.dense_tensor_product(M, Drot @ x, Drot @ y)
        rhs = Drot @ cg_tensor.dense_tensor_product(M, x, y)
        np.testing.assert_allclose(lhs, rhs, atol=1e-11)
