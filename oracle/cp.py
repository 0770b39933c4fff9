"""CP decomposition of the CG tensor and its error metrics.

Naming.  The paper writes M_kij ~ sum_r A_kr B_ir C_jr (Sec. 3.1, eq. cp)
with A on the output mode, B on the first operand x and C on the second
operand y.  Here those are called D (output, [d3, R]), A (x, [d1, R]) and
B (y, [d2, R]), so eq. approximate reads m(x, y) ~ D (A^T x  (*)  B^T y).

* ``cp_als``: rank-R fit by alternating least squares (the paper names ALS
  or gradient methods, Sec. 3.4, and fits once and caches the factors,
  Sec. 4.1).  Each factor in turn solves its normal equations, whose Gram
  matrix is the elementwise product of the other two factors' Grams; then the
  columns of A and B are normalised and the norms moved into D.
* ``universality_factors``: the exact rank-d1*d2 construction of Thm. 2
  (App. B.2): column r = (i, j) has A = e_i, B = e_j, D = M[:, i, j].
* ``approximation_error`` / ``equivariance_error`` / ``equivariance_bound``:
  the metrics of Sec. 4.1 and the intermediate inequality in the proof of
  Thm. 1 (eq. derive_upper_bound), eps <= 2 ||M - M_hat||_F ||x|| ||y||.
* ``tucker_tail`` / ``hosvd_truncate``: the mode-n singular-value tail of
  Thm. 1 with R_T = floor(R^(1/3)), and the truncated HOSVD it bounds.
"""
from __future__ import annotations

import numpy as np

from .cg_tensor import dense_tensor_product


def cp_reconstruct(D: np.ndarray, A: np.ndarray, B: np.ndarray) -> np.ndarray:
    """M_hat[k, i, j] = sum_r D[k,r] A[i,r] B[j,r]."""
    return np.einsum("kr,ir,jr->kij", D, A, B)


def cp_apply(D, A, B, x, y):
    """eq. approximate: D (A^T x  (*)  B^T y); x: [..., d1], y: [..., d2]."""
    return (((x @ A) * (y @ B)) @ D.T)


def _khatri_rao(U: np.ndarray, V: np.ndarray) -> np.ndarray:
    """Column-wise Kronecker product, rows ordered (u, v) with v fastest."""
    return (U[:, None, :] * V[None, :, :]).reshape(U.shape[0] * V.shape[0], U.shape[1])


def _solve(mttkrp: np.ndarray, gram: np.ndarray, ridge: float) -> np.ndarray:
    g = gram + ridge * np.mean(np.diag(gram)) * np.eye(gram.shape[0])
    return np.linalg.solve(g, mttkrp.T).T


def cp_als(M: np.ndarray, R: int, seed: int, max_sweeps: int = 2000, tol: float = 1e-12,
           ridge: float = 1e-10, history: list | None = None):
    """One seeded ALS run.  Returns (D, A, B, relative Frobenius error)."""
    d3, d1, d2 = M.shape
    rng = np.random.default_rng(seed)
    A = rng.normal(size=(d1, R))
    B = rng.normal(size=(d2, R))
    D = rng.normal(size=(d3, R))
    M1 = M.reshape(d3, d1 * d2)                       # rows k, cols (i, j)
    M2 = M.transpose(1, 0, 2).reshape(d1, d3 * d2)    # rows i, cols (k, j)
    M3 = M.transpose(2, 0, 1).reshape(d2, d3 * d1)    # rows j, cols (k, i)
    norm = np.linalg.norm(M)
    prev = np.inf
    err = np.inf
    for _ in range(max_sweeps):
        D = _solve(M1 @ _khatri_rao(A, B), (A.T @ A) * (B.T @ B), ridge)
        A = _solve(M2 @ _khatri_rao(D, B), (D.T @ D) * (B.T @ B), ridge)
        nA = np.linalg.norm(A, axis=0)
        nA[nA == 0] = 1.0
        A /= nA
        D *= nA
        B = _solve(M3 @ _khatri_rao(D, A), (D.T @ D) * (A.T @ A), ridge)
        nB = np.linalg.norm(B, axis=0)
        nB[nB == 0] = 1.0
        B /= nB
        D *= nB
        err = np.linalg.norm(M - cp_reconstruct(D, A, B)) / norm
        if history is not None:
            history.append(err)
        if abs(prev - err) < tol:
            break
        prev = err
    return D, A, B, float(err)


def cp_fit(M: np.ndarray, R: int, seed: int, restarts: int = 3, **kw):
    """Best of ``restarts`` seeded ALS runs (seeds seed, seed+1, ...)."""
    best = None
    for s in range(restarts):
        res = cp_als(M, R, seed + s, **kw)
        if best is None or res[3] < best[3]:
            best = res
    return best


def universality_factors(M: np.ndarray):
    """Thm. 2: exact CP factors with R = d1 * d2 (column r = i * d2 + j)."""
    d3, d1, d2 = M.shape
    A = np.zeros((d1, d1 * d2))
    B = np.zeros((d2, d1 * d2))
    D = np.zeros((d3, d1 * d2))
    for i in range(d1):
        for j in range(d2):
            r = i * d2 + j
            A[i, r] = 1.0
            B[j, r] = 1.0
            D[:, r] = M[:, i, j]
    return D, A, B


def approximation_error(M, D, A, B, x, y) -> np.ndarray:
    """||M(x(x)y) - M_hat(x(x)y)|| / ||M(x(x)y)|| per sample (Sec. 4.1)."""
    ref = dense_tensor_product(M, x, y)
    app = cp_apply(D, A, B, x, y)
    return np.linalg.norm(ref - app, axis=-1) / np.linalg.norm(ref, axis=-1)


def equivariance_error(D, A, B, Drot: np.ndarray, x, y) -> np.ndarray:
    """eps(R, x, y) = ||M_hat(D(R)x (x) D(R)y) - D(R) M_hat(x (x) y)|| (Sec. 3.4)."""
    lhs = cp_apply(D, A, B, x @ Drot.T, y @ Drot.T)
    rhs = cp_apply(D, A, B, x, y) @ Drot.T
    return np.linalg.norm(lhs - rhs, axis=-1)


def equivariance_bound(M, D, A, B, x, y) -> np.ndarray:
    """2 ||M - M_hat||_F ||x|| ||y|| (proof of Thm. 1, eq. derive_upper_bound)."""
    diff = np.linalg.norm(M - cp_reconstruct(D, A, B))
    return 2.0 * diff * np.linalg.norm(x, axis=-1) * np.linalg.norm(y, axis=-1)


def unfold(M: np.ndarray, n: int) -> np.ndarray:
    return np.moveaxis(M, n, 0).reshape(M.shape[n], -1)


def tucker_tail(M: np.ndarray, R: int) -> float:
    """(sum_n sum_{k > R_T} sigma_k^(n)^2)^(1/2) with R_T = floor(R^(1/3))."""
    RT = int(np.floor(R ** (1.0 / 3.0) + 1e-12))
    tot = 0.0
    for n in range(3):
        s = np.linalg.svd(unfold(M, n), compute_uv=False)
        tot += float(np.sum(s[RT:] ** 2))
    return float(np.sqrt(tot))


def hosvd_truncate(M: np.ndarray, rank: int) -> np.ndarray:
    """Truncated higher-order SVD with multilinear rank (rank, rank, rank)."""
    Us = []
    for n in range(3):
        U, _, _ = np.linalg.svd(unfold(M, n), full_matrices=False)
        Us.append(U[:, :rank])
    core = np.einsum("kij,ka,ib,jc->abc", M, Us[0], Us[1], Us[2])
    return np.einsum("abc,ka,ib,jc->kij", core, Us[0], Us[1], Us[2])
