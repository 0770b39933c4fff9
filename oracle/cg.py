"""Clebsch-Gordan coefficients and their real-basis form.

The CG tensor product of two irreps (Sec. 2, eq. clebsch_gordan) couples a
degree-l1 and a degree-l2 feature into every degree l3 with
|l1 - l2| <= l3 <= l1 + l2 through the coefficients C^{l3 m3}_{l1 m1 l2 m2}.

* ``cg_complex`` evaluates them in the standard complex (Condon-Shortley)
  basis with Racah's closed formula, summed in exact rational arithmetic.
* ``complex_to_real`` is the unitary Q_l with Y_real = sqrt(4 pi) Q_l Y_complex
  for the real basis of ``oracle.sh`` (no Condon-Shortley phase in the real
  functions; component normalisation is the sqrt(4 pi)).
* ``cg_real`` is the block C_real[m3, m1, m2] in that real basis: with
  x_real = Q x_complex for every feature,
      C_real = sum Q3[m3,u3] C[u3,u1,u2] conj(Q1[m1,u1]) conj(Q2[m2,u2]).
  It comes out purely real, or purely imaginary when l1 + l2 + l3 is odd; an
  imaginary block is multiplied by -i (any real multiple of an equivariant
  map is equivariant, so this fixes only a sign convention).
"""
from __future__ import annotations

from fractions import Fraction
from functools import lru_cache
from math import factorial, sqrt

import numpy as np


def _f(n: int) -> int:
    return factorial(n)


@lru_cache(maxsize=None)
def cg_complex(j1: int, m1: int, j2: int, m2: int, J: int, M: int) -> float:
    """<j1 m1; j2 m2 | J M> by Racah's formula (integer degrees)."""
    if M != m1 + m2:
        return 0.0
    if not (abs(j1 - j2) <= J <= j1 + j2):
        return 0.0
    if abs(m1) > j1 or abs(m2) > j2 or abs(M) > J:
        return 0.0
    pref = Fraction((2 * J + 1) * _f(J + j1 - j2) * _f(J - j1 + j2) * _f(j1 + j2 - J),
                    _f(j1 + j2 + J + 1))
    pref *= _f(J + M) * _f(J - M) * _f(j1 - m1) * _f(j1 + m1) * _f(j2 - m2) * _f(j2 + m2)
    s = Fraction(0)
    for k in range(0, j1 + j2 - J + 1):
        args = (k, j1 + j2 - J - k, j1 - m1 - k, j2 + m2 - k, J - j2 + m1 + k, J - j1 - m2 + k)
        if min(args) < 0:
            continue
        den = 1
        for a in args:
            den *= _f(a)
        s += Fraction((-1) ** k, den)
    if s == 0:
        return 0.0
    sq = pref * s * s                      # exact square of the coefficient
    return (1.0 if s > 0 else -1.0) * sqrt(sq.numerator / sq.denominator)


@lru_cache(maxsize=None)
def complex_to_real(l: int) -> np.ndarray:
    """Q_l, rows = real order m, columns = complex order u, both -l..l.

    m > 0:  Y_real[m]  = (Y_c[-m] + (-1)^m Y_c[m]) / sqrt(2)
    m < 0:  Y_real[m]  = i (Y_c[m] - (-1)^|m| Y_c[|m|]) / sqrt(2)
    m = 0:  Y_real[0]  = Y_c[0]
    (each times sqrt(4 pi)), from Re/Im of Y_c[|m|] and
    conj(Y_c[u]) = (-1)^u Y_c[-u]."""
    n = 2 * l + 1
    Q = np.zeros((n, n), dtype=np.complex128)
    s = 1.0 / sqrt(2.0)
    Q[l, l] = 1.0
    for m in range(1, l + 1):
        Q[l + m, l - m] = s
        Q[l + m, l + m] = (-1) ** m * s
        Q[l - m, l - m] = 1j * s
        Q[l - m, l + m] = -1j * (-1) ** m * s
    Q.setflags(write=False)
    return Q


def cg_complex_block(l1: int, l2: int, l3: int) -> np.ndarray:
    """C[u3, u1, u2] in the complex basis, shape [2l3+1, 2l1+1, 2l2+1]."""
    out = np.zeros((2 * l3 + 1, 2 * l1 + 1, 2 * l2 + 1))
    for u1 in range(-l1, l1 + 1):
        for u2 in range(-l2, l2 + 1):
            u3 = u1 + u2
            if abs(u3) <= l3:
                out[u3 + l3, u1 + l1, u2 + l2] = cg_complex(l1, u1, l2, u2, l3, u3)
    return out


@lru_cache(maxsize=None)
def cg_real(l1: int, l2: int, l3: int) -> np.ndarray:
    """Real-basis CG block C_real[m3, m1, m2] (orthonormal: sum of squares
    equals 2 l3 + 1)."""
    C = cg_complex_block(l1, l2, l3)
    Q1, Q2, Q3 = complex_to_real(l1), complex_to_real(l2), complex_to_real(l3)
    Cr = np.einsum("au,uvw,bv,cw->abc", Q3, C, Q1.conj(), Q2.conj())
    if (l1 + l2 + l3) % 2:
        Cr = -1j * Cr
    assert np.max(np.abs(Cr.imag)) < 1e-12, "real-basis CG block is not real"
    out = np.ascontiguousarray(Cr.real)
    out.setflags(write=False)
    return out
