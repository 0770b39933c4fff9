"""The CG coefficient tensor M over all admissible paths, and the dense tensor
product it defines.

Sec. 2: a path is a triple (l1, l2, l3) with |l1 - l2| <= l3 <= l1 + l2; the
full tensor product up to degree L keeps the paths with l1, l2 <= L and
l3 <= min(l1 + l2, L).  Sec. 3.1: M is the direct sum of the CG blocks of
those paths, a three-way tensor in R^{d3 x d1 x d2} with d = (L+1)^2 for all
three modes, and the bilinear map is m(x, y)_k = sum_ij M_kij x_i y_j
(eq. bilinear).  Index order: k = (l3, m3) output, i = (l1, m1) first operand,
j = (l2, m2) second operand, each flattened as l*l + l + m.  Every path enters
with coefficient 1 (no parity filter).
"""
from __future__ import annotations

from functools import lru_cache

import numpy as np

from .cg import cg_real


def paths(L: int) -> list[tuple[int, int, int]]:
    return [(l1, l2, l3)
            for l1 in range(L + 1) for l2 in range(L + 1)
            for l3 in range(abs(l1 - l2), min(l1 + l2, L) + 1)]


@lru_cache(maxsize=None)
def cg_tensor(L: int) -> np.ndarray:
    """M[k, i, j], shape [(L+1)^2]*3, float64."""
    d = (L + 1) ** 2
    M = np.zeros((d, d, d))
    for l1, l2, l3 in paths(L):
        M[l3 * l3:(l3 + 1) ** 2, l1 * l1:(l1 + 1) ** 2, l2 * l2:(l2 + 1) ** 2] = cg_real(l1, l2, l3)
    M.setflags(write=False)
    return M


def dense_tensor_product(M: np.ndarray, x: np.ndarray, y: np.ndarray) -> np.ndarray:
    """m(x, y) = M(x (x) y): sum_ij M_kij x_i y_j (eq. bilinear).

    x: [..., d1], y: [..., d2] -> [..., d3]."""
    return np.einsum("kij,...i,...j->...k", M, x, y)
