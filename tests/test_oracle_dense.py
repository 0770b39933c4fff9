"""Pins of the exact CG tensor-product layer (oracle/dense_layer.py): it is the
CP layer of oracle/layer.py for an exact factorisation whose ranks each lie in
one path (Thm. 2), it reduces to a closed form on a single path, and it is
rotation equivariant."""
import numpy as np
import pytest

import workloads
from oracle import cg_tensor, dense_layer, layer, sh, wigner


def _graph(seed, L, P, N=12, E=90, C=8):
    return workloads.random_graph(seed, n_nodes=N, n_edges=E, L=L, C=C, R=P)


@pytest.mark.parametrize("L", [0, 1, 2, 3])
def test_equals_the_cp_layer_with_exact_per_path_factors(L):
    P = len(cg_tensor.paths(L))
    w = _graph(40 + L, L, P)
    D, A, B, rank_path = dense_layer.exact_cp_factors(L)
    # the factorisation is exact: sum_r D[:, r] A[i, r] B[j, r] = M
    np.testing.assert_allclose(np.einsum("kr,ir,jr->kij", D, A, B), cg_tensor.cg_tensor(L), atol=1e-15)
    radial_cp = w["radial_w"][:, rank_path]         # rank r carries the weight of its path
    want = layer.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], radial_cp, w["r_cut"], L)
    got, Z = dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], w["W"], w["radial_w"], w["r_cut"], L,
                                 return_z=True)
    assert np.max(np.abs(got - want)) < 1e-12 * max(1.0, np.max(np.abs(want)))
    np.testing.assert_allclose(Z @ np.asarray(w["W"], np.float64), got, rtol=0, atol=1e-12)


def test_single_path_zero_l_l_is_scalar_times_harmonics():
    # C[l m3; 0 0, l m2] = delta(m2, m3) in the real basis, so the path (0, l, l)
    # alone gives z_e^(l) = rho_e x[s]^(0) Y_e^(l) and zero in every other degree
    L, l = 3, 2
    plist = cg_tensor.paths(L)
    P = len(plist)
    w = _graph(7, L, P)
    pw = np.zeros_like(w["radial_w"], dtype=np.float64)
    pw[:, plist.index((0, l, l))] = w["radial_w"][:, 0]
    _, Z = dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], w["W"], pw, w["r_cut"], L, return_z=True)
    vec = w["edge_vec"].astype(np.float64)
    Y = sh.spherical_harmonics(L, vec)
    phi, _ = layer.radial_basis(np.linalg.norm(vec, axis=1), w["r_cut"], pw.shape[0])
    rho = phi @ pw[:, plist.index((0, l, l))]
    s, t = w["edge_index"]
    want = np.zeros_like(Z)
    for e in range(len(s)):
        want[t[e], l * l:(l + 1) ** 2, :] += rho[e] * Y[e, l * l:(l + 1) ** 2, None] * w["x"][s[e], 0, None, :]
    np.testing.assert_allclose(Z, want, rtol=0, atol=1e-12)


@pytest.mark.parametrize("L", [1, 2, 4])
def test_rotation_equivariance(L):
    P = len(cg_tensor.paths(L))
    w = _graph(60 + L, L, P, C=4)
    Rm = wigner.random_rotation(np.random.default_rng(L))
    Dr = wigner.wigner_d_full(L, Rm)
    out = dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], w["W"], w["radial_w"], w["r_cut"], L)
    x2 = np.einsum("ab,nbc->nac", Dr, w["x"].astype(np.float64))
    out2 = dense_layer.forward(x2, w["edge_index"], w["edge_vec"].astype(np.float64) @ Rm.T, w["W"],
                               w["radial_w"], w["r_cut"], L)
    np.testing.assert_allclose(out2, np.einsum("ab,nbc->nac", Dr, out), rtol=0, atol=1e-10 * np.max(np.abs(out)))


@pytest.mark.parametrize("L", [2, 4])
def test_path_index_covers_exactly_the_nonzero_coefficients(L):
    M = cg_tensor.cg_tensor(L)
    Pi = dense_layer.path_index(L)
    assert np.all(Pi[M != 0] >= 0)
    # the blocks of distinct paths never overlap: every (k, i, j) has one path
    count = np.zeros(M.shape, np.int64)
    for l1, l2, l3 in cg_tensor.paths(L):
        count[l3 * l3:(l3 + 1) ** 2, l1 * l1:(l1 + 1) ** 2, l2 * l2:(l2 + 1) ** 2] += 1
    assert count.max() == 1


# ----- the product without path-weight sharing (one W_p per path)

def _wpaths(seed, P, C):
    rng = np.random.default_rng(seed)
    return rng.normal(size=(P, C, C)) / np.sqrt(C)


@pytest.mark.parametrize("L", [0, 1, 2, 3])
def test_unshared_with_equal_path_weights_is_the_shared_product(L):
    P = len(cg_tensor.paths(L))
    w = _graph(80 + L, L, P)
    Wp = np.repeat(np.asarray(w["W"], np.float64)[None], P, axis=0)
    got = dense_layer.forward_unshared(w["x"], w["edge_index"], w["edge_vec"], Wp, w["radial_w"], w["r_cut"], L)
    want = dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], w["W"], w["radial_w"], w["r_cut"], L)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12 * max(1.0, np.max(np.abs(want))))


def test_unshared_is_the_sum_of_single_path_products_each_with_its_own_weight():
    # linear in the paths: switching all but one path off (its radial weight)
    # leaves that path's product with its own W_p; the sum over paths of those
    # single-path shared products is the unshared product
    L = 2
    plist = cg_tensor.paths(L)
    P = len(plist)
    w = _graph(91, L, P)
    Wp = _wpaths(3, P, w["C"])
    total = dense_layer.forward_unshared(w["x"], w["edge_index"], w["edge_vec"], Wp, w["radial_w"], w["r_cut"], L)
    acc = np.zeros_like(total)
    for p in range(P):
        pw = np.zeros_like(w["radial_w"], dtype=np.float64)
        pw[:, p] = w["radial_w"][:, p]
        acc += dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], Wp[p], pw, w["r_cut"], L)
    np.testing.assert_allclose(total, acc, rtol=0, atol=1e-12 * np.max(np.abs(total)))


def test_unshared_single_path_zero_l_l_closed_form():
    # only the path (0, l, l) on: m_e^(l) = rho_e Y_e^(l) (x[s]^(0) W_p), other degrees zero
    L, l = 3, 2
    plist = cg_tensor.paths(L)
    P = len(plist)
    p0 = plist.index((0, l, l))
    w = _graph(17, L, P)
    pw = np.zeros_like(w["radial_w"], dtype=np.float64)
    pw[:, p0] = w["radial_w"][:, 0]
    Wp = _wpaths(5, P, w["C"])
    out = dense_layer.forward_unshared(w["x"], w["edge_index"], w["edge_vec"], Wp, pw, w["r_cut"], L)
    vec = w["edge_vec"].astype(np.float64)
    Y = sh.spherical_harmonics(L, vec)
    phi, _ = layer.radial_basis(np.linalg.norm(vec, axis=1), w["r_cut"], pw.shape[0])
    rho = phi @ pw[:, p0]
    s, t = w["edge_index"]
    want = np.zeros_like(out)
    for e in range(len(s)):
        want[t[e], l * l:(l + 1) ** 2, :] += rho[e] * Y[e, l * l:(l + 1) ** 2, None] * (
            np.asarray(w["x"][s[e], 0], np.float64) @ Wp[p0])[None, :]
    np.testing.assert_allclose(out, want, rtol=0, atol=1e-12 * np.max(np.abs(want)))


@pytest.mark.parametrize("L", [1, 3])
def test_unshared_rotation_equivariance(L):
    P = len(cg_tensor.paths(L))
    w = _graph(70 + L, L, P, C=4)
    Wp = _wpaths(L, P, 4)
    Rm = wigner.random_rotation(np.random.default_rng(10 + L))
    Dr = wigner.wigner_d_full(L, Rm)
    out = dense_layer.forward_unshared(w["x"], w["edge_index"], w["edge_vec"], Wp, w["radial_w"], w["r_cut"], L)
    x2 = np.einsum("ab,nbc->nac", Dr, w["x"].astype(np.float64))
    out2 = dense_layer.forward_unshared(x2, w["edge_index"], w["edge_vec"].astype(np.float64) @ Rm.T, Wp,
                                        w["radial_w"], w["r_cut"], L)
    np.testing.assert_allclose(out2, np.einsum("ab,nbc->nac", Dr, out), rtol=0,
                               atol=1e-10 * np.max(np.abs(out)))
