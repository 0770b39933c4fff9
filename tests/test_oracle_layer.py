"""Pins for the oracle's message-passing layer (oracle/layer.py).

Independent references: with the exact factors of Thm. 2 and a radial weight
that is one scalar per edge, the layer is the dense CG product summed over
edges, computed here by brute-force contraction of M; that layer is then
exactly equivariant under rotations; linearity identities; a single edge is
one evaluation of eq. approximate; finite differences for every gradient;
numpy's stable argsort for the edge order."""
import numpy as np
import pytest

import workloads
from oracle import cg_tensor, cp, layer, sh, wigner


def _factors(L, R, seed):
    rng = np.random.default_rng(seed)
    d = (L + 1) ** 2
    A, B, D = rng.normal(size=(3, d, R)) / np.sqrt(d)
    return A, B, D


def test_stable_sort_matches_numpy_and_offsets():
    rng = np.random.default_rng(0)
    for n, e in [(10, 0), (1, 17), (50, 400), (7, 1000)]:
        key = rng.integers(0, n, size=e)
        perm, off = layer.stable_sort_by_key(key, n)
        np.testing.assert_array_equal(perm, np.argsort(key, kind="stable"))
        np.testing.assert_array_equal(off, np.concatenate([[0], np.cumsum(np.bincount(key, minlength=n))]))
        assert off[-1] == e and np.all(np.diff(off) >= 0)


def test_radial_basis_closed_form_and_derivative():
    rc, n = 6.0, 8
    mu = np.arange(n) * rc / (n - 1)
    phi, _ = layer.radial_basis(mu, rc, n)
    np.testing.assert_allclose(np.diag(phi), 1.0)
    np.testing.assert_allclose(phi[0, 1], np.exp(-0.5))
    r = np.linspace(0.5, 5.5, 11)
    _, dphi = layer.radial_basis(r, rc, n)
    h = 1e-6
    fd = (layer.radial_basis(r + h, rc, n)[0] - layer.radial_basis(r - h, rc, n)[0]) / (2 * h)
    np.testing.assert_allclose(dphi, fd, rtol=1e-7, atol=1e-9)


def test_tiny_layer_matches_einsum_reduction():
    w = workloads.random_graph(3, n_nodes=6, n_edges=20, L=1, C=3, R=5)
    A, B, D = _factors(1, 5, 0)
    out = layer.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"],
                        w["r_cut"], 1)
    Y = sh.spherical_harmonics(1, w["edge_vec"].astype(np.float64))
    phi, _ = layer.radial_basis(np.linalg.norm(w["edge_vec"].astype(np.float64), axis=1), w["r_cut"], 8)
    rho = phi @ w["radial_w"]
    s, t = w["edge_index"]
    m = np.einsum("kr,ir,jr,eic,ej,er,cf->ekf", D, A, B, w["x"][s].astype(np.float64), Y, rho,
                  w["W"].astype(np.float64))
    ref = np.zeros_like(out)
    np.add.at(ref, t, m)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


def _scalar_radial(R, seed):
    """radial weight matrix with identical columns: rho_e is one scalar per edge."""
    col = np.random.default_rng(seed).normal(size=(8, 1))
    return np.repeat(col, R, axis=1)


@pytest.mark.parametrize("L", [1, 2])
def test_exact_factors_reproduce_dense_cg_layer(L):
    M = cg_tensor.cg_tensor(L)
    D, A, B = cp.universality_factors(M)
    R = D.shape[1]
    w = workloads.random_graph(11 + L, n_nodes=9, n_edges=40, L=L, C=4, R=R)
    Wrad = _scalar_radial(R, L)
    out = layer.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], Wrad, w["r_cut"], L)
    vec = w["edge_vec"].astype(np.float64)
    Y = sh.spherical_harmonics(L, vec)
    phi, _ = layer.radial_basis(np.linalg.norm(vec, axis=1), w["r_cut"], 8)
    rho = (phi @ Wrad)[:, 0]
    s, t = w["edge_index"]
    ref = np.zeros_like(out)
    x = w["x"].astype(np.float64)
    for e in range(w["E"]):            # brute-force dense contraction per edge
        msg = np.einsum("kij,ic,j->kc", M, x[s[e]], Y[e]) * rho[e]
        ref[t[e]] += msg @ w["W"].astype(np.float64)
    np.testing.assert_allclose(out, ref, rtol=1e-12, atol=1e-12)


def test_exact_factors_layer_is_equivariant():
    L = 2
    M = cg_tensor.cg_tensor(L)
    D, A, B = cp.universality_factors(M)
    R = D.shape[1]
    w = workloads.random_graph(21, n_nodes=8, n_edges=30, L=L, C=3, R=R)
    Wrad = _scalar_radial(R, 2)
    rng = np.random.default_rng(9)
    Rm = wigner.random_rotation(rng)
    Drot = wigner.wigner_d_full(L, Rm)
    args = (w["edge_index"],)
    out = layer.forward(w["x"], *args, w["edge_vec"], A, B, D, w["W"], Wrad, w["r_cut"], L)
    xr = np.einsum("ab,nbc->nac", Drot, w["x"].astype(np.float64))
    vr = w["edge_vec"].astype(np.float64) @ Rm.T
    out_r = layer.forward(xr, *args, vr, A, B, D, w["W"], Wrad, w["r_cut"], L)
    np.testing.assert_allclose(out_r, np.einsum("ab,nbc->nac", Drot, out), atol=1e-11)


def test_single_edge_is_one_cp_product():
    L, R, C = 3, 12, 5
    A, B, D = _factors(L, R, 4)
    w = workloads.random_graph(5, n_nodes=2, n_edges=1, L=L, C=C, R=R)
    w["edge_index"][:] = np.array([[0], [1]])
    x = w["x"].astype(np.float64)
    out = layer.forward(x, w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], w["r_cut"], L)
    vec = w["edge_vec"][0].astype(np.float64)
    y = sh.spherical_harmonics(L, vec)
    phi, _ = layer.radial_basis(np.array([np.linalg.norm(vec)]), w["r_cut"], 8)
    rho = (phi @ w["radial_w"])[0]
    # eq. approximate per channel c, times the radial weight on the rank index, then W
    msg = np.stack([D @ ((A.T @ x[0][:, c]) * (B.T @ y) * rho) for c in range(C)], 1)
    np.testing.assert_allclose(out[1], msg @ w["W"], rtol=1e-12, atol=1e-12)
    np.testing.assert_array_equal(out[0], 0)


def _problem(seed=31, L=2, R=7, C=4, N=6, E=25):
    A, B, D = _factors(L, R, seed)
    w = workloads.random_graph(seed, n_nodes=N, n_edges=E, L=L, C=C, R=R)
    f = {k: np.asarray(w[k], np.float64) for k in ("x", "W", "radial_w", "grad_out", "edge_vec")}
    return A, B, D, w, f


def test_linearity_identities():
    A, B, D, w, f = _problem()
    L = 2
    out = layer.forward(f["x"], w["edge_index"], f["edge_vec"], A, B, D, f["W"], f["radial_w"], w["r_cut"], L)
    gx, gW, _ = layer.backward(f["x"], w["edge_index"], f["edge_vec"], A, B, D, f["W"], f["radial_w"],
                               w["r_cut"], L, f["grad_out"])
    s = np.sum(f["grad_out"] * out)
    assert abs(np.sum(gx * f["x"]) - s) < 1e-10 * max(1, abs(s))
    assert abs(np.sum(gW * f["W"]) - s) < 1e-10 * max(1, abs(s))


def test_backward_finite_differences():
    A, B, D, w, f = _problem()
    L = 2
    ei = w["edge_index"]

    def loss(x=None, W=None, vec=None, Wr=None):
        o = layer.forward(f["x"] if x is None else x, ei, f["edge_vec"] if vec is None else vec, A, B, D,
                          f["W"] if W is None else W, f["radial_w"] if Wr is None else Wr, w["r_cut"], L)
        return np.sum(o * f["grad_out"])

    gx, gW, gv, gr = layer.backward(f["x"], ei, f["edge_vec"], A, B, D, f["W"], f["radial_w"], w["r_cut"], L,
                                    f["grad_out"], return_radial=True)
    h = 1e-6
    rng = np.random.default_rng(0)
    assert gr.shape == f["radial_w"].shape
    for q in range(gr.shape[0]):
        for r in range(0, gr.shape[1], 5):
            Rp, Rm = f["radial_w"].astype(np.float64), f["radial_w"].astype(np.float64)
            Rp[q, r] += h
            Rm[q, r] -= h
            fd = (loss(Wr=Rp) - loss(Wr=Rm)) / (2 * h)
            assert abs(fd - gr[q, r]) < 1e-6 * max(1, abs(gr[q, r])), (q, r, fd, gr[q, r])
    for _ in range(6):
        idx = tuple(rng.integers(0, s) for s in f["x"].shape)
        xp, xm = f["x"].copy(), f["x"].copy()
        xp[idx] += h
        xm[idx] -= h
        assert abs((loss(x=xp) - loss(x=xm)) / (2 * h) - gx[idx]) < 1e-6 * max(1, abs(gx[idx]))
        idx = tuple(rng.integers(0, s) for s in f["W"].shape)
        Wp, Wm = f["W"].copy(), f["W"].copy()
        Wp[idx] += h
        Wm[idx] -= h
        assert abs((loss(W=Wp) - loss(W=Wm)) / (2 * h) - gW[idx]) < 1e-6 * max(1, abs(gW[idx]))
    for e in range(w["E"]):
        for a in range(3):
            vp, vm = f["edge_vec"].copy(), f["edge_vec"].copy()
            vp[e, a] += h
            vm[e, a] -= h
            fd = (loss(vec=vp) - loss(vec=vm)) / (2 * h)
            assert abs(fd - gv[e, a]) < 1e-6 * max(1, abs(gv[e, a])), (e, a, fd, gv[e, a])


def test_sampled_forward_matches_full():
    A, B, D, w, f = _problem(seed=41, N=12, E=60)
    L = 2
    out = layer.forward(f["x"], w["edge_index"], f["edge_vec"], A, B, D, f["W"], f["radial_w"], w["r_cut"], L)
    nodes = np.array([0, 5, 11])
    sub = layer.forward_at_nodes(nodes, f["x"], w["edge_index"], f["edge_vec"], A, B, D, f["W"],
                                 f["radial_w"], w["r_cut"], L)
    np.testing.assert_array_equal(sub, out[nodes])


# ------------------------------------------------------------ three-input product (App. A)
def _tp3_graph(seed, L, R, N=10, E=60, C=3):
    return workloads.random_graph(seed, n_nodes=N, n_edges=E, L=L, C=C, R=R)


def test_three_input_with_constant_third_factor_is_the_two_input_layer():
    # A2 = e_0 (one in the degree-0 row) and x[:, 0, :] = 1 make A2^T x[t] = 1
    L, R = 2, 6
    w = _tp3_graph(1, L, R)
    rng = np.random.default_rng(2)
    A, B, D = (rng.normal(size=((L + 1) ** 2, R)) for _ in range(3))
    x = np.array(w["x"], np.float64)
    x[:, 0, :] = 1.0
    A2 = np.zeros_like(A)
    A2[0, :] = 1.0
    got = layer.forward3(x, w["edge_index"], w["edge_vec"], A, A2, B, D, w["W"], w["radial_w"], w["r_cut"], L)
    want = layer.forward(x, w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], w["r_cut"], L)
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12 * np.max(np.abs(want)))


def _cg3_factors(L):
    """Exact CP factors of T[k, i, j, l] = sum_m M[k, m, l] M[m, i, j], the
    trilinear map M(M(x, y), z): one rank per (i, j, l)."""
    M = cg_tensor.cg_tensor(L)
    T = np.einsum("kml,mij->kijl", M, M)
    d = M.shape[0]
    idx = [(i, j, l) for i in range(d) for j in range(d) for l in range(d) if np.any(T[:, i, j, l] != 0)]
    A = np.zeros((d, len(idx)))
    B = np.zeros((d, len(idx)))
    A2 = np.zeros((d, len(idx)))
    D = np.zeros((d, len(idx)))
    for r, (i, j, l) in enumerate(idx):
        A[i, r] = B[j, r] = A2[l, r] = 1.0
        D[:, r] = T[:, i, j, l]
    return T, A, A2, B, D


def test_three_input_exact_factors_give_the_nested_cg_product_and_equivariance():
    L = 1
    T, A, A2, B, D = _cg3_factors(L)
    R = A.shape[1]
    w = _tp3_graph(3, L, R)
    rw = np.repeat(np.random.default_rng(4).normal(size=(8, 1)), R, axis=1)   # one radial weight per edge
    got = layer.forward3(w["x"], w["edge_index"], w["edge_vec"], A, A2, B, D, w["W"], rw, w["r_cut"], L)
    vec = w["edge_vec"].astype(np.float64)
    Y = sh.spherical_harmonics(L, vec)
    phi, _ = layer.radial_basis(np.linalg.norm(vec, axis=1), w["r_cut"], 8)
    rho = (phi @ rw)[:, 0]
    s, t = w["edge_index"]
    x = w["x"].astype(np.float64)
    # brute force: M(M(x[s], Y), x[t]) channel by channel, scaled by rho
    M = cg_tensor.cg_tensor(L)
    inner = np.einsum("mij,eic,ej->emc", M, x[s], Y)
    msg = np.einsum("kml,emc,elc->ekc", M, inner, x[t]) * rho[:, None, None]
    want = np.zeros_like(got)
    np.add.at(want, t, msg @ w["W"].astype(np.float64))
    np.testing.assert_allclose(got, want, rtol=0, atol=1e-12 * np.max(np.abs(want)))
    Rm = wigner.random_rotation(np.random.default_rng(5))
    Dr = wigner.wigner_d_full(L, Rm)
    x2 = np.einsum("ab,nbc->nac", Dr, x)
    got2 = layer.forward3(x2, w["edge_index"], vec @ Rm.T, A, A2, B, D, w["W"], rw, w["r_cut"], L)
    np.testing.assert_allclose(got2, np.einsum("ab,nbc->nac", Dr, got), rtol=0, atol=1e-10 * np.max(np.abs(got)))


# ------------------------------------------------------------ path-weight-shared linear layer
def test_ps_linear_identity_scaling_and_equivariance():
    rng = np.random.default_rng(8)
    L, C = 3, 5
    d = (L + 1) ** 2
    x = rng.normal(size=(7, d, C))
    np.testing.assert_allclose(layer.ps_linear(x, np.eye(C), L), x, rtol=0, atol=0)
    np.testing.assert_allclose(layer.ps_linear(x, 2.5 * np.eye(C), L), 2.5 * x, rtol=1e-15)
    W = rng.normal(size=(C, C))
    y = layer.ps_linear(x, W, L)
    # it acts on channels only, so it commutes with every Wigner-D rotation
    Dr = wigner.wigner_d_full(L, wigner.random_rotation(rng))
    y2 = layer.ps_linear(np.einsum("ab,nbc->nac", Dr, x), W, L)
    np.testing.assert_allclose(y2, np.einsum("ab,nbc->nac", Dr, y), rtol=0, atol=1e-12)
    # one channel vector at a time: column f of y is x's channels against W[:, f]
    for f in range(C):
        np.testing.assert_allclose(y[..., f], np.tensordot(x, W[:, f], axes=([2], [0])), rtol=1e-13)
