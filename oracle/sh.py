"""Real spherical harmonics from the closed form of the regular solid harmonics.

The paper only names the spherical harmonics of the edge direction as the
second operand of the tensor product (Sec. 1, Sec. 2); the convention used
here is:

* degree l = 0..L, order m = -l..l, flat index l*l + l + m, so d = (L+1)^2;
* real basis without the Condon-Shortley phase, z is the polar axis:
  m > 0 takes Re((x + i y)^m), m < 0 takes Im((x + i y)^|m|);
* "component" normalisation: Y_00 = 1 and sum_m Y_lm(u)^2 = 2l + 1 on the
  unit sphere.

Regular solid harmonic (homogeneous polynomial of degree l):
    S_lm(r) = sqrt(2l+1) * N_l|m| * P_m(x, y) * Lambda_l^|m|(z, r^2)
    N_lm    = sqrt((2 - delta_m0) (l-m)! / (l+m)!)
    Lambda_l^m(z, r^2) = 2^-l sum_k (-1)^k C(l,k) C(2l-2k,l) (l-2k)!/(l-2k-m)!
                          * (r^2)^k z^(l-2k-m),   k = 0 .. floor((l-m)/2)
and Y_lm(u) = S_lm(u) for unit u.
"""
from __future__ import annotations

from math import comb, factorial, sqrt

import numpy as np


def n_components(L: int) -> int:
    return (L + 1) ** 2


def index(l: int, m: int) -> int:
    return l * l + l + m


def _lambda_terms(l: int, m: int):
    """Coefficients of Lambda_l^m as a list of (coef, k, zpow)."""
    out = []
    for k in range((l - m) // 2 + 1):
        c = ((-1) ** k) * comb(l, k) * comb(2 * l - 2 * k, l) * factorial(l - 2 * k) \
            / factorial(l - 2 * k - m) / 2.0 ** l
        out.append((c, k, l - 2 * k - m))
    return out


def _xy_power(x, y, m):
    """(Re, Im) of (x + i y)^m by repeated complex multiplication."""
    re = np.ones_like(x)
    im = np.zeros_like(x)
    for _ in range(m):
        re, im = re * x - im * y, re * y + im * x
    return re, im


def solid_harmonics(L: int, r: np.ndarray) -> np.ndarray:
    """S_lm(r) for all l <= L.  r: [..., 3] float64 -> [..., (L+1)^2]."""
    r = np.asarray(r, dtype=np.float64)
    x, y, z = r[..., 0], r[..., 1], r[..., 2]
    r2 = x * x + y * y + z * z
    out = np.zeros(r.shape[:-1] + (n_components(L),))
    for l in range(L + 1):
        for m in range(0, l + 1):
            lam = np.zeros_like(x)
            for c, k, zp in _lambda_terms(l, m):
                lam = lam + c * r2 ** k * z ** zp
            norm = sqrt(2 * l + 1) * sqrt((2 - (m == 0)) * factorial(l - m) / factorial(l + m))
            re, im = _xy_power(x, y, m)
            out[..., index(l, m)] = norm * re * lam
            if m > 0:
                out[..., index(l, -m)] = norm * im * lam
    return out


def solid_harmonics_grad(L: int, r: np.ndarray) -> np.ndarray:
    """Gradient dS_lm/dr.  r: [..., 3] -> [..., (L+1)^2, 3].

    Product rule on P_m(x, y) * Lambda(z, r^2), using
      d/dx (x+iy)^m = m (x+iy)^(m-1),  d/dy (x+iy)^m = i m (x+iy)^(m-1),
      d/dx (r^2)^k  = 2k (r^2)^(k-1) x  (likewise y, z)."""
    r = np.asarray(r, dtype=np.float64)
    x, y, z = r[..., 0], r[..., 1], r[..., 2]
    r2 = x * x + y * y + z * z
    out = np.zeros(r.shape[:-1] + (n_components(L), 3))
    for l in range(L + 1):
        for m in range(0, l + 1):
            lam = np.zeros_like(x)
            dlam = np.zeros(r.shape)            # gradient of Lambda
            for c, k, zp in _lambda_terms(l, m):
                lam = lam + c * r2 ** k * z ** zp
                if k > 0:
                    g = c * 2 * k * r2 ** (k - 1) * z ** zp
                    dlam[..., 0] += g * x
                    dlam[..., 1] += g * y
                    dlam[..., 2] += g * z
                if zp > 0:
                    dlam[..., 2] += c * r2 ** k * zp * z ** (zp - 1)
            norm = sqrt(2 * l + 1) * sqrt((2 - (m == 0)) * factorial(l - m) / factorial(l + m))
            re, im = _xy_power(x, y, m)
            if m > 0:
                re1, im1 = _xy_power(x, y, m - 1)
            else:
                re1, im1 = np.zeros_like(x), np.zeros_like(x)
            # gradient of Re/Im (x+iy)^m
            d_re = np.stack([m * re1, -m * im1, np.zeros_like(x)], -1)
            d_im = np.stack([m * im1, m * re1, np.zeros_like(x)], -1)
            out[..., index(l, m), :] = norm * (d_re * lam[..., None] + re[..., None] * dlam)
            if m > 0:
                out[..., index(l, -m), :] = norm * (d_im * lam[..., None] + im[..., None] * dlam)
    return out


def spherical_harmonics(L: int, vec: np.ndarray) -> np.ndarray:
    """Y(vec/|vec|) for all l <= L.  vec: [..., 3] -> [..., (L+1)^2]."""
    vec = np.asarray(vec, dtype=np.float64)
    u = vec / np.linalg.norm(vec, axis=-1, keepdims=True)
    return solid_harmonics(L, u)


def spherical_harmonics_jacobian(L: int, vec: np.ndarray) -> np.ndarray:
    """dY(vec/|vec|)/dvec  -> [..., (L+1)^2, 3].

    S_lm is homogeneous of degree l, so Y(vec) = S(vec)/|vec|^l and
      dY/dvec = (grad S(u) - l S(u) u) / |vec|,  u = vec/|vec|."""
    vec = np.asarray(vec, dtype=np.float64)
    n = np.linalg.norm(vec, axis=-1, keepdims=True)
    u = vec / n
    S = solid_harmonics(L, u)
    dS = solid_harmonics_grad(L, u)
    ls = np.concatenate([np.full(2 * l + 1, l) for l in range(L + 1)]).astype(np.float64)
    jac = dS - (ls[:, None] * S[..., :, None]) * u[..., None, :]
    return jac / n[..., None]
