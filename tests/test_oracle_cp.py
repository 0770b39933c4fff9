"""Pins for the oracle's CP decomposition and error metrics (oracle/cp.py).

Independent references: exact recovery of a synthetic rank-R tensor, the
monotone residual of unregularised ALS, the exact construction of Thm. 2,
the inequality in the proof of Thm. 1, and the truncated-HOSVD bound."""
import numpy as np
import pytest

from oracle import cg_tensor, cp, wigner


def test_als_recovers_exact_low_rank_tensor():
    rng = np.random.default_rng(0)
    d, R = 9, 5
    Dt, At, Bt = rng.normal(size=(3, d, R))
    T = cp.cp_reconstruct(Dt, At, Bt)
    D, A, B, err = cp.cp_fit(T, R, seed=3, restarts=3, max_sweeps=3000, ridge=1e-14, tol=0)
    assert err < 1e-7
    np.testing.assert_allclose(cp.cp_reconstruct(D, A, B), T, atol=1e-6)


def test_als_residual_non_increasing_without_ridge():
    M = cg_tensor.cg_tensor(2)
    hist = []
    cp.cp_als(M, 16, seed=1, max_sweeps=150, ridge=1e-14, tol=0, history=hist)
    assert np.all(np.diff(hist) <= 1e-12)
    assert hist[-1] < hist[0]


def test_full_rank_fit_is_exact_at_rank_d_squared_bound():
    # generic bound rank_CP(M) <= min(d1 d2, d1 d3, d2 d3) (Sec. 3.3)
    M = cg_tensor.cg_tensor(1)
    D, A, B, err = cp.cp_fit(M, 16, seed=0, restarts=2, max_sweeps=3000, ridge=1e-14, tol=0)
    assert err < 1e-6


@pytest.mark.parametrize("L", [1, 2, 3])
def test_universality_construction_is_exact(L):
    M = cg_tensor.cg_tensor(L)
    D, A, B = cp.universality_factors(M)
    d = (L + 1) ** 2
    assert D.shape[1] == d * d
    np.testing.assert_array_equal(cp.cp_reconstruct(D, A, B), M)
    rng = np.random.default_rng(L)
    x, y = rng.normal(size=(2, 7, d))
    np.testing.assert_allclose(cp.cp_apply(D, A, B, x, y), cg_tensor.dense_tensor_product(M, x, y),
                               atol=1e-13)
    Drot = wigner.wigner_d_full(L, wigner.random_rotation(rng))
    assert np.max(cp.equivariance_error(D, A, B, Drot, x, y)) < 1e-12


def test_equivariance_bound_holds_for_fitted_factors():
    L, R = 2, 16
    M = cg_tensor.cg_tensor(L)
    D, A, B, err = cp.cp_als(M, R, seed=0, max_sweeps=300)
    assert 0 < err < 1
    rng = np.random.default_rng(5)
    d = (L + 1) ** 2
    x, y = rng.normal(size=(2, 100, d))
    x /= np.linalg.norm(x, axis=1, keepdims=True)
    y /= np.linalg.norm(y, axis=1, keepdims=True)
    bound = cp.equivariance_bound(M, D, A, B, x, y)
    worst = 0.0
    for _ in range(20):
        Drot = wigner.wigner_d_full(L, wigner.random_rotation(rng))
        eps = cp.equivariance_error(D, A, B, Drot, x, y)
        assert np.all(eps <= bound + 1e-12)
        worst = max(worst, float(np.max(eps / bound)))
    assert worst > 1e-3          # the fit is not equivariant by accident
    app = cp.approximation_error(M, D, A, B, x, y)
    assert np.all(app >= 0) and np.mean(app) < 1.0


@pytest.mark.parametrize("L,R", [(2, 8), (2, 27), (3, 64)])
def test_hosvd_truncation_within_tail_bound(L, R):
    M = cg_tensor.cg_tensor(L)
    RT = int(np.floor(R ** (1 / 3) + 1e-12))
    trunc = cp.hosvd_truncate(M, RT)
    assert np.linalg.norm(M - trunc) <= cp.tucker_tail(M, R) + 1e-12


def test_tucker_tail_vanishes_at_full_multilinear_rank():
    M = cg_tensor.cg_tensor(1)
    assert cp.tucker_tail(M, 4 ** 3) < 1e-12


# ----- approximation_error (Sec. 4.1): closed-form cases that fix both the
# numerator and the normaliser.  A normaliser taken from the approximation
# instead of the exact product, or squared norms, fails each of them.

@pytest.mark.parametrize("L", [1, 2, 3])
def test_approximation_error_zero_for_exact_factors(L):
    # Thm. 2: the rank d^2 construction reproduces M, so the error is 0
    M = cg_tensor.cg_tensor(L)
    D, A, B = cp.universality_factors(M)
    rng = np.random.default_rng(10 + L)
    x, y = rng.normal(size=(2, 50, (L + 1) ** 2))
    app = cp.approximation_error(M, D, A, B, x, y)
    assert np.max(app) < 1e-14


@pytest.mark.parametrize("L", [1, 2])
def test_approximation_error_one_for_zero_approximation(L):
    M = cg_tensor.cg_tensor(L)
    D, A, B = cp.universality_factors(M)
    rng = np.random.default_rng(20 + L)
    x, y = rng.normal(size=(2, 30, (L + 1) ** 2))
    app = cp.approximation_error(M, np.zeros_like(D), A, B, x, y)
    np.testing.assert_array_equal(app, np.ones(30))


@pytest.mark.parametrize("eps", [0.5, -0.25, 1e-3, 3.0])
def test_approximation_error_of_scaled_tensor_is_abs_eps(eps):
    # M_hat = (1 + eps) M  =>  error = |eps| for every sample; the
    # approximation's norm as normaliser would give |eps| / |1 + eps|, and
    # squared norms eps^2
    M = cg_tensor.cg_tensor(2)
    D, A, B = cp.universality_factors(M)
    rng = np.random.default_rng(7)
    x, y = rng.normal(size=(2, 40, 9))
    app = cp.approximation_error(M, (1.0 + eps) * D, A, B, x, y)
    np.testing.assert_allclose(app, abs(eps), rtol=1e-12)


def test_approximation_error_hand_computed_degree_one_case():
    # L = 1 (d = 4).  The path 0 x 1 -> 1 has the identity as its CG block
    # (<0 0; 1 m' | 1 m> = delta), so with x the unit scalar e_0 the exact
    # product is M(e_0 (x) y) = y.  Dropping that path from the Thm. 2 factors
    # (zeroing the columns (i = 0, j in degree 1)) leaves (y_0, 0, 0, 0).
    # With y = (3, 0, 4, 0): error = ||(0, 0, 4, 0)|| / ||y|| = 4 / 5 exactly
    # (the approximation's norm would give 4/3, squared norms 16/25).
    M = cg_tensor.cg_tensor(1)
    D, A, B = cp.universality_factors(M)
    x = np.array([[1.0, 0.0, 0.0, 0.0]])
    y = np.array([[3.0, 0.0, 4.0, 0.0]])
    np.testing.assert_allclose(cg_tensor.dense_tensor_product(M, x, y), y, atol=1e-15)
    D2 = D.copy()
    for j in (1, 2, 3):
        D2[:, 0 * 4 + j] = 0.0
    app = cp.approximation_error(M, D2, A, B, x, y)
    np.testing.assert_allclose(app, [0.8], rtol=1e-14)
