"""The exact (dense) CG tensor-product message-passing layer, path by path --
TEST INFRASTRUCTURE ONLY (the comparator of the CP layer in oracle/layer.py).

Sec. 2 (eq. clebsch_gordan and the complete product over all paths): for every
path (l1, l2, l3) with l1, l2 <= L and |l1 - l2| <= l3 <= min(l1 + l2, L), the
degree-l3 block of x (x)_CG y is sum over m1, m2 of C[l3 m3; l1 m1, l2 m2]
x^(l1)_m1 y^(l2)_m2.  Sec. 3.2: in the unshared product each path carries its
own weight; here that weight is a radial function of the edge,

    rho_e[p] = phi_e Wpath[:, p]       (phi_e the Gaussian basis of |r_e|)

and the multiplicity (channel) weight W is the one matrix all paths share
(path-weight sharing; equal columns of Wpath make the radial weight shared
too).  For every edge e = (s, t):

    Y_e    = Y(r_e / |r_e|)
    z_e^(l3) = sum over paths p = (l1, l2, l3) of
               rho_e[p] * sum_{m1, m2} C[l3 m3; l1 m1, l2 m2] x[s]^(l1)_m1 Y_e^(l2)_m2
    Z[t]  = sum over edges into t of z_e        (in sorted-edge order)
    out   = Z W

The path list is cg_tensor.paths(L) in its order (the index p of Wpath);
the CG blocks are cg.cg_real, the same real-basis blocks that build M.
Float64 throughout.

``forward_unshared`` is the product without path-weight sharing (the fully
connected CG tensor product of Sec. 3.2, whose O(L^3) paths each carry a
distinct multiplicity-space weight): per edge and path the degree-l3 block
rho_e[p] CG_p(x[s], Y_e) is multiplied by that path's own channel matrix
W_p [C_in, C_out] before the paths are summed,

    m_e^(l3) = sum over paths p = (l1, l2, l3) of
               (rho_e[p] * sum_{m1, m2} C[l3 m3; l1 m1, l2 m2] x[s]^(l1)_m1 Y_e^(l2)_m2) W_p,

so that W_p = W for every p is the shared product above.
"""
from __future__ import annotations

import numpy as np

from .cg import cg_real
from .cg_tensor import paths
from .layer import radial_basis, stable_sort_by_key
from .sh import spherical_harmonics


def forward(x, edge_index, edge_vec, W, path_w, r_cut, L, perm=None, return_z=False):
    """out [N, d, C] (and Z, the per-node sum before W, when return_z)."""
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    path_w = np.asarray(path_w, np.float64)
    N, d, C = x.shape
    plist = paths(L)
    assert path_w.shape[1] == len(plist)
    src = np.asarray(edge_index[0], np.int64)
    dst = np.asarray(edge_index[1], np.int64)
    if perm is None:
        perm, _ = stable_sort_by_key(dst, N)
    perm = np.asarray(perm, np.int64)
    vec = np.asarray(edge_vec, np.float64)[perm]
    Y = spherical_harmonics(L, vec)                                   # [E, d]
    phi, _ = radial_basis(np.linalg.norm(vec, axis=1), r_cut, path_w.shape[0])
    rho = phi @ path_w                                                # [E, P]
    xs = x[src[perm]]                                                 # [E, d, C]
    z = np.zeros((perm.shape[0], d, C))
    for p, (l1, l2, l3) in enumerate(plist):
        blk = cg_real(l1, l2, l3)                                     # [2l3+1, 2l1+1, 2l2+1]
        a = slice(l1 * l1, (l1 + 1) ** 2)
        b = slice(l2 * l2, (l2 + 1) ** 2)
        o = slice(l3 * l3, (l3 + 1) ** 2)
        z[:, o, :] += rho[:, p, None, None] * np.einsum("kij,eic,ej->ekc", blk, xs[:, a, :], Y[:, b])
    Z = np.zeros((N, d, C))
    np.add.at(Z, dst[perm], z)                                        # in sorted order
    out = Z @ W
    return (out, Z) if return_z else out


def forward_unshared(x, edge_index, edge_vec, W_paths, path_w, r_cut, L, perm=None):
    """out [N, d, C] of the product with one channel matrix per path,
    W_paths [P, C_in, C_out], applied to each edge's path block before the
    paths and the edges are summed (in sorted-edge order)."""
    x = np.asarray(x, np.float64)
    W_paths = np.asarray(W_paths, np.float64)
    path_w = np.asarray(path_w, np.float64)
    N, d, C = x.shape
    plist = paths(L)
    assert path_w.shape[1] == len(plist) and W_paths.shape[0] == len(plist)
    src = np.asarray(edge_index[0], np.int64)
    dst = np.asarray(edge_index[1], np.int64)
    if perm is None:
        perm, _ = stable_sort_by_key(dst, N)
    perm = np.asarray(perm, np.int64)
    vec = np.asarray(edge_vec, np.float64)[perm]
    Y = spherical_harmonics(L, vec)
    phi, _ = radial_basis(np.linalg.norm(vec, axis=1), r_cut, path_w.shape[0])
    rho = phi @ path_w
    xs = x[src[perm]]
    m = np.zeros((perm.shape[0], d, W_paths.shape[2]))
    for p, (l1, l2, l3) in enumerate(plist):
        blk = cg_real(l1, l2, l3)
        a = slice(l1 * l1, (l1 + 1) ** 2)
        b = slice(l2 * l2, (l2 + 1) ** 2)
        o = slice(l3 * l3, (l3 + 1) ** 2)
        zp = rho[:, p, None, None] * np.einsum("kij,eic,ej->ekc", blk, xs[:, a, :], Y[:, b])
        m[:, o, :] += zp @ W_paths[p]
    out = np.zeros((N, d, W_paths.shape[2]))
    np.add.at(out, dst[perm], m)                                      # in sorted order
    return out


def exact_cp_factors(L):
    """Thm. 2's construction refined by output degree: one rank per
    (i, j, l3) with a nonzero CG block entry, A[i, r] = B[j, r] = 1 and
    D[k, r] = M[k, i, j] for k in degree l3 only, so that each rank lies in
    exactly one path.  Returns D, A, B and the path index of every rank."""
    d = (L + 1) ** 2
    index = {pth: p for p, pth in enumerate(paths(L))}
    cols_D, cols_A, cols_B, rank_path = [], [], [], []
    for (l1, l2, l3), p in index.items():
        blk = cg_real(l1, l2, l3)
        for mi in range(2 * l1 + 1):
            for mj in range(2 * l2 + 1):
                col = blk[:, mi, mj]
                if not np.any(col != 0.0):
                    continue
                i, j = l1 * l1 + mi, l2 * l2 + mj
                dcol = np.zeros(d)
                dcol[l3 * l3:(l3 + 1) ** 2] = col
                cols_D.append(dcol)
                cols_A.append(np.eye(d)[i])
                cols_B.append(np.eye(d)[j])
                rank_path.append(p)
    return (np.stack(cols_D, 1), np.stack(cols_A, 1), np.stack(cols_B, 1), np.asarray(rank_path, np.int64))


def path_index(L):
    """P[k, i, j]: the index in paths(L) of the path whose CG block holds
    entry (k, i, j) of M, -1 outside every block."""
    d = (L + 1) ** 2
    P = -np.ones((d, d, d), np.int64)
    for p, (l1, l2, l3) in enumerate(paths(L)):
        P[l3 * l3:(l3 + 1) ** 2, l1 * l1:(l1 + 1) ** 2, l2 * l2:(l2 + 1) ** 2] = p
    return P

