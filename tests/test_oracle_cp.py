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
