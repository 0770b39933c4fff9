"""Real Wigner-D matrices: the representation D(R) of a rotation R in the real
spherical-harmonic basis (used in Sec. 3.4 to define the equivariance error
and in the proof of Thm. 1, App. B.1).

Two independent constructions:

* ``wigner_d_from_sh``: D_l(R) is the unique matrix with
  Y_l(R u) = D_l(R) Y_l(u) for every unit u; it is solved by least squares
  from the closed-form harmonics at 4(2l+1) random points.
* ``wigner_d_euler``: Wigner's closed formula for the small-d matrix,
  D^l_{m'm}(a, b, c) = e^{-i m' a} d^l_{m'm}(b) e^{-i m c} for
  R = Rz(a) Ry(b) Rz(c), taken to the real basis with the unitary Q_l of
  ``oracle.cg``.  With the complex harmonics satisfying
  Y_c(R^-1 u) = D(R)^T Y_c(u) (the standard convention for this formula),
  the real matrix is  Q conj(D(R)) Q^H.

Random rotations come from normalised seeded Gaussian quaternions, which are
uniform on SO(3).
"""
from __future__ import annotations

from math import factorial, sqrt

import numpy as np

from .cg import complex_to_real
from .sh import solid_harmonics


def random_rotation(rng: np.random.Generator) -> np.ndarray:
    q = rng.normal(size=4)
    q /= np.linalg.norm(q)
    w, x, y, z = q
    return np.array([[1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
                     [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
                     [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)]])


def wigner_d_from_sh(l: int, R: np.ndarray, seed: int = 0) -> np.ndarray:
    rng = np.random.default_rng(seed)
    u = rng.normal(size=(4 * (2 * l + 1), 3))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    sl = slice(l * l, (l + 1) ** 2)
    Y = solid_harmonics(l, u)[:, sl]                  # [n, 2l+1]
    YR = solid_harmonics(l, u @ R.T)[:, sl]           # Y(R u)
    # YR = Y D^T  ->  D^T = lstsq(Y, YR)
    Dt, *_ = np.linalg.lstsq(Y, YR, rcond=None)
    return Dt.T


def wigner_d_full(L: int, R: np.ndarray, seed: int = 0) -> np.ndarray:
    """Block-diagonal D(R) over degrees 0..L, shape [(L+1)^2, (L+1)^2]."""
    d = (L + 1) ** 2
    out = np.zeros((d, d))
    for l in range(L + 1):
        sl = slice(l * l, (l + 1) ** 2)
        out[sl, sl] = wigner_d_from_sh(l, R, seed)
    return out


def euler_zyz(R: np.ndarray) -> tuple[float, float, float]:
    """(a, b, c) with R = Rz(a) Ry(b) Rz(c)."""
    b = np.arccos(np.clip(R[2, 2], -1.0, 1.0))
    if abs(np.sin(b)) > 1e-12:
        a = np.arctan2(R[1, 2], R[0, 2])
        c = np.arctan2(R[2, 1], -R[2, 0])
    else:
        a = np.arctan2(R[1, 0], R[0, 0]) if R[2, 2] > 0 else np.arctan2(-R[1, 0], -R[0, 0])
        c = 0.0
    return float(a), float(b), float(c)


def small_d(l: int, b: float) -> np.ndarray:
    """Wigner small-d matrix d^l_{m'm}(b), rows m', columns m (Wigner's sum)."""
    n = 2 * l + 1
    out = np.zeros((n, n))
    cb, sb = np.cos(b / 2), np.sin(b / 2)
    for mp in range(-l, l + 1):
        for m in range(-l, l + 1):
            pre = sqrt(factorial(l + mp) * factorial(l - mp) * factorial(l + m) * factorial(l - m))
            s = 0.0
            for k in range(max(0, m - mp), min(l + m, l - mp) + 1):
                s += ((-1) ** (mp - m + k) * cb ** (2 * l + m - mp - 2 * k) * sb ** (mp - m + 2 * k)
                      / (factorial(l + m - k) * factorial(k) * factorial(mp - m + k)
                         * factorial(l - mp - k)))
            out[mp + l, m + l] = pre * s
    return out


def wigner_d_euler(l: int, R: np.ndarray) -> np.ndarray:
    a, b, c = euler_zyz(R)
    ms = np.arange(-l, l + 1)
    Dc = np.exp(-1j * ms[:, None] * a) * small_d(l, b) * np.exp(-1j * ms[None, :] * c)
    Q = complex_to_real(l)
    Dr = Q @ Dc.conj() @ Q.conj().T
    assert np.max(np.abs(Dr.imag)) < 1e-10
    return Dr.real


def rot_z(a):
    c, s = np.cos(a), np.sin(a)
    return np.array([[c, -s, 0], [s, c, 0], [0, 0, 1.0]])


def rot_y(b):
    c, s = np.cos(b), np.sin(b)
    return np.array([[c, 0, s], [0, 1.0, 0], [-s, 0, c]])


