"""Seeded synthetic atomic geometries and radius graphs.

Nothing here computes any part of the CP tensor-product layer: this module
only places atoms and lists the directed neighbour pairs within a cutoff, the
way the layer's callers would.  The geometries stand in for the paper's
workloads (organic molecules of PubChemQCR, catalyst slabs with adsorbates of
OC20/OC22, Sec. 4 "Datasets"), which are not available here.

Conventions
-----------
* Positions are in Angstrom, float64 while generated.
* An edge e is a directed pair (src, dst) with 0 < |r_e| < r_cut strictly and
  src != dst; both directions of every pair are present.
* The edge vector is r_e = pos[src] - pos[dst] (+ the periodic image shift).
* Periodic axes use the minimum image; cell lengths are at least 2 r_cut along
  every periodic axis, so at most one image of any pair is within r_cut.
"""
from __future__ import annotations

import numpy as np


def _random_unit(rng: np.random.Generator) -> np.ndarray:
    v = rng.normal(size=3)
    return v / np.linalg.norm(v)


def molecule_walk(rng: np.random.Generator, n_atoms: int, bond: float = 1.5,
                  sphere: float = 3.5, clash: float = 1.2,
                  ring_start: bool = False, jitter: float = 0.3) -> np.ndarray:
    """A chain/ring molecule grown as a self-avoiding random walk.

    Each new atom sits one bond length from the previous atom in a uniform
    random direction, stays within ``sphere`` of atom 0 and keeps at least
    ``clash`` from every earlier atom other than its bonded predecessor.
    With ``ring_start`` the first six atoms form a planar hexagon.  Every
    coordinate is finally jittered by U(-jitter, +jitter).
    """
    pos = []
    if ring_start:
        ang = np.arange(6) * (np.pi / 3.0)
        # regular hexagon with side = bond, random orientation
        ring = np.stack([bond * np.cos(ang), bond * np.sin(ang), np.zeros(6)], 1)
        q = rng.normal(size=4)
        q /= np.linalg.norm(q)
        w, x, y, z = q
        rot = np.array([[1 - 2 * (y * y + z * z), 2 * (x * y - z * w), 2 * (x * z + y * w)],
                        [2 * (x * y + z * w), 1 - 2 * (x * x + z * z), 2 * (y * z - x * w)],
                        [2 * (x * z - y * w), 2 * (y * z + x * w), 1 - 2 * (x * x + y * y)]])
        ring = ring @ rot.T
        ring -= ring[0]
        pos.extend(list(ring[: min(6, n_atoms)]))
    else:
        pos.append(np.zeros(3))
    attempts = 0
    while len(pos) < n_atoms:
        attempts += 1
        if attempts > 200000:
            raise RuntimeError("molecule_walk: could not place atoms")
        # grow from the last atom; after repeated failures, branch from a random atom
        anchor = len(pos) - 1 if attempts % 50 else int(rng.integers(len(pos)))
        cand = pos[anchor] + bond * _random_unit(rng)
        if np.linalg.norm(cand - pos[0]) > sphere:
            continue
        arr = np.asarray(pos)
        dist = np.linalg.norm(arr - cand, axis=1)
        dist[anchor] = np.inf
        if np.all(dist >= clash):
            pos.append(cand)
    arr = np.asarray(pos, dtype=np.float64)
    arr += rng.uniform(-jitter, jitter, size=arr.shape)
    return arr


def fcc_slab(rng: np.random.Generator, a: float = 3.6, nx: int = 5, ny: int = 5,
             nz: int = 3, noise: float = 0.1) -> tuple[np.ndarray, np.ndarray]:
    """fcc lattice of nx*ny*nz conventional cells (4 atoms each) with Gaussian
    noise; returns (positions, cell lengths (Lx, Ly))."""
    basis = np.array([[0, 0, 0], [0.5, 0.5, 0], [0.5, 0, 0.5], [0, 0.5, 0.5]])
    cells = np.array([[i, j, k] for i in range(nx) for j in range(ny) for k in range(nz)],
                     dtype=np.float64)
    pos = (cells[:, None, :] + basis[None, :, :]).reshape(-1, 3) * a
    pos += rng.normal(scale=noise, size=pos.shape)
    return pos, np.array([nx * a, ny * a])


def random_sequential_addition(rng: np.random.Generator, n_atoms: int, box: float,
                               min_sep: float = 1.0) -> np.ndarray:
    """Uniform random points in a periodic cube, rejecting any point closer
    than ``min_sep`` (minimum image) to an accepted one."""
    pos = np.empty((n_atoms, 3))
    n = 0
    tries = 0
    while n < n_atoms:
        tries += 1
        if tries > 100 * n_atoms:
            raise RuntimeError("random_sequential_addition: too dense")
        cand = rng.uniform(0.0, box, size=3)
        if n:
            dv = pos[:n] - cand
            dv -= box * np.round(dv / box)
            if np.min(np.einsum("ij,ij->i", dv, dv)) < min_sep * min_sep:
                continue
        pos[n] = cand
        n += 1
    return pos


def radius_graph(pos: np.ndarray, r_cut: float, cell: np.ndarray | None = None,
                 periodic: tuple[bool, bool, bool] = (False, False, False),
                 chunk: int = 1024) -> tuple[np.ndarray, np.ndarray, np.ndarray]:
    """All directed pairs (src, dst), src != dst, with |pos[src]-pos[dst]| < r_cut.

    Returns (src, dst, vec) with vec = pos[src] - pos[dst] after the minimum
    image along periodic axes, sorted by (dst, src).
    """
    n = pos.shape[0]
    per = np.asarray(periodic, dtype=bool)
    if per.any():
        cell = np.asarray(cell, dtype=np.float64)
        assert np.all(cell[per] >= 2 * r_cut), "cell too small for minimum image"
    srcs, dsts, vecs = [], [], []
    for d0 in range(0, n, chunk):
        d1 = min(n, d0 + chunk)
        dv = pos[None, :, :] - pos[d0:d1, None, :]          # [nd, n, 3] = pos[src]-pos[dst]
        if per.any():
            dv[..., per] -= cell[per] * np.round(dv[..., per] / cell[per])
        dist2 = np.einsum("abk,abk->ab", dv, dv)
        ok = dist2 < r_cut * r_cut
        ok[np.arange(d1 - d0), np.arange(d0, d1)] = False
        di, si = np.nonzero(ok)                              # row-major: sorted by (dst, src)
        srcs.append(si)
        dsts.append(di + d0)
        vecs.append(dv[di, si])
    src = np.concatenate(srcs).astype(np.int64)
    dst = np.concatenate(dsts).astype(np.int64)
    vec = np.concatenate(vecs)
    return src, dst, vec
