"""The CP tensor-product message-passing layer by literal per-edge summation.

For every edge e = (s, t) with vector r_e (Sec. 3.1 eq. approximate with
y = Y(r_e / |r_e|), Sec. 3.2 path-weight sharing):

    Y_e   = Y(r_e / |r_e|)                         real spherical harmonics
    phi_e = exp(-(|r_e| - mu_q)^2 / (2 sigma^2)),  q = 0..n_radial-1,
            mu_q = q r_cut / (n_radial - 1),  sigma = r_cut / (n_radial - 1)
    rho_e = phi_e Wrad                              radial weight per rank
    v_e   = B^T Y_e                                 second-operand projection
    g_e   = v_e * rho_e
    u_e   = A^T x[s]          ([R, C], per channel)  first-operand projection
    h_e   = diag(g_e) u_e                           Hadamard product
    z_e   = D h_e             ([d, C])               output factor
    m_e   = z_e W             ([d, C])               one W shared by all paths
    out[t] = sum over edges into t of m_e           (in sorted-edge order)

Everything is float64 from the exact stored input values.  D and W are applied
per edge, as written; nothing is reassociated.  The backward is the chain rule
through the same per-edge steps (factors A, B, D are constants, Sec. 4.1).
"""
from __future__ import annotations

import numpy as np

from .sh import spherical_harmonics, spherical_harmonics_jacobian

CHUNK = 256


# ----------------------------------------------------------------- sorting
def stable_sort_by_key(key: np.ndarray, n_keys: int):
    """Stable counting sort of edge ids by key (dst for the forward, src for
    the transposed graph).  Returns (perm, offsets): perm[p] is the original
    edge id in sorted slot p, offsets[k] the first slot of key k,
    offsets[n_keys] = E."""
    key = np.asarray(key, dtype=np.int64)
    counts = np.zeros(n_keys + 1, dtype=np.int64)
    for k in key:
        counts[k + 1] += 1
    offsets = np.cumsum(counts)
    nxt = offsets[:-1].copy()
    perm = np.empty(key.shape[0], dtype=np.int64)
    for e, k in enumerate(key):          # original order -> stable
        perm[nxt[k]] = e
        nxt[k] += 1
    return perm.astype(np.int32), offsets.astype(np.int32)


# ----------------------------------------------------------------- geometry
def radial_basis(dist: np.ndarray, r_cut: float, n_radial: int):
    """Gaussian radial basis phi [E, n] and its derivative dphi/d|r|."""
    mu = np.arange(n_radial) * (r_cut / (n_radial - 1))
    sigma = r_cut / (n_radial - 1)
    diff = dist[:, None] - mu[None, :]
    phi = np.exp(-diff * diff / (2.0 * sigma * sigma))
    dphi = -diff / (sigma * sigma) * phi
    return phi, dphi


def edge_terms(edge_vec, L, B, radial_w, r_cut):
    """Y [E,d], phi [E,n], rho [E,R], v [E,R], g [E,R] for every edge."""
    vec = np.asarray(edge_vec, dtype=np.float64)
    Y = spherical_harmonics(L, vec)
    phi, _ = radial_basis(np.linalg.norm(vec, axis=1), r_cut, radial_w.shape[0])
    rho = phi @ np.asarray(radial_w, np.float64)
    v = Y @ np.asarray(B, np.float64)
    return Y, phi, rho, v, v * rho


def _f64(*arrs):
    return [np.asarray(a, dtype=np.float64) for a in arrs]


# ----------------------------------------------------------------- forward
def forward(x, edge_index, edge_vec, A, B, D, W, radial_w, r_cut, L,
            perm=None, return_z=False):
    """out [N, d, C] (and optionally the per-node sum of z_e, the tensor the
    layer has before W, for checking the saved activation)."""
    x, A, B, D, W = _f64(x, A, B, D, W)
    N, d, C = x.shape
    src = np.asarray(edge_index[0], np.int64)
    dst = np.asarray(edge_index[1], np.int64)
    if perm is None:
        perm, _ = stable_sort_by_key(dst, N)
    perm = np.asarray(perm, np.int64)
    out = np.zeros((N, d, C))
    zsum = np.zeros((N, d, C)) if return_z else None
    for c0 in range(0, perm.shape[0], CHUNK):
        ids = perm[c0:c0 + CHUNK]
        _, _, _, _, g = edge_terms(np.asarray(edge_vec)[ids], L, B, radial_w, r_cut)
        u = np.matmul(A.T[None], x[src[ids]])              # [e, R, C]
        h = g[:, :, None] * u
        z = np.matmul(D[None], h)                          # [e, d, C]
        m = z @ W
        np.add.at(out, dst[ids], m)                        # in sorted order
        if return_z:
            np.add.at(zsum, dst[ids], z)
    return (out, zsum) if return_z else out


def ps_linear(x, W, L):
    """The equivariant linear layer with path-weight sharing (Sec. 3.2; used
    for the linear layers, Sec. 4.1): for every degree l the block
    x^(l) [N, 2l+1, C] is multiplied by the one channel matrix W, degree by
    degree as the per-degree layer would be with all W_l equal."""
    x = np.asarray(x, np.float64)
    W = np.asarray(W, np.float64)
    y = np.zeros(x.shape[:2] + (W.shape[1],))
    for l in range(L + 1):
        blk = slice(l * l, (l + 1) ** 2)
        y[:, blk, :] = np.einsum("nmc,cf->nmf", x[:, blk, :], W)
    return y


def forward3(x, edge_index, edge_vec, A, A2, B, D, W, radial_w, r_cut, L, perm=None):
    """The three-input product (App. A, eq. multi-tp with N = 3 and its CP
    form D (B1^T x1 * B2^T x2 * B3^T x3)), the inputs being the source node's
    features, the edge's harmonics and the destination node's features:
    per edge e = (s, t),  h_e = g_e * (A^T x[s]) * (A2^T x[t]),  z_e = D h_e,
    m_e = z_e W,  out[t] = sum of m_e (sorted order).  Float64."""
    x, A, A2, B, D, W = _f64(x, A, A2, B, D, W)
    N, d, C = x.shape
    src = np.asarray(edge_index[0], np.int64)
    dst = np.asarray(edge_index[1], np.int64)
    if perm is None:
        perm, _ = stable_sort_by_key(dst, N)
    perm = np.asarray(perm, np.int64)
    out = np.zeros((N, d, C))
    for c0 in range(0, perm.shape[0], CHUNK):
        ids = perm[c0:c0 + CHUNK]
        _, _, _, _, g = edge_terms(np.asarray(edge_vec)[ids], L, B, radial_w, r_cut)
        u = np.matmul(A.T[None], x[src[ids]])              # [e, R, C]
        u2 = np.matmul(A2.T[None], x[dst[ids]])            # [e, R, C]
        h = g[:, :, None] * u * u2
        z = np.matmul(D[None], h)
        np.add.at(out, dst[ids], z @ W)
    return out


# ----------------------------------------------------------------- backward
def backward(x, edge_index, edge_vec, A, B, D, W, radial_w, r_cut, L, grad_out,
             perm=None, return_radial=False):
    """Returns (grad_x [N,d,C], grad_W [C,C], grad_edge_vec [E,3]) for the
    scalar <grad_out, out>, and with return_radial also grad_radial_w
    [n_radial, R] (rho_e = phi_e Wrad, so dL/dWrad = sum_e phi_e^T drho_e)."""
    x, A, B, D, W, G = _f64(x, A, B, D, W, grad_out)
    Wrad = np.asarray(radial_w, np.float64)
    N, d, C = x.shape
    src = np.asarray(edge_index[0], np.int64)
    dst = np.asarray(edge_index[1], np.int64)
    E = src.shape[0]
    if perm is None:
        perm, _ = stable_sort_by_key(dst, N)
    perm = np.asarray(perm, np.int64)
    grad_x = np.zeros_like(x)
    grad_W = np.zeros((C, C))
    grad_vec = np.zeros((E, 3))
    grad_wrad = np.zeros_like(Wrad)
    for c0 in range(0, E, CHUNK):
        ids = perm[c0:c0 + CHUNK]
        vec = np.asarray(edge_vec, np.float64)[ids]
        Y, phi, rho, v, g = edge_terms(vec, L, B, Wrad, r_cut)
        dist = np.linalg.norm(vec, axis=1)
        _, dphi = radial_basis(dist, r_cut, Wrad.shape[0])
        u = np.matmul(A.T[None], x[src[ids]])              # [e, R, C]
        h = g[:, :, None] * u
        z = np.matmul(D[None], h)                          # [e, d, C]
        Gt = G[dst[ids]]                                   # dL/dm_e  [e, d, C]
        grad_W += np.einsum("edc,edf->cf", z, Gt)          # m = z W
        Gz = Gt @ W.T                                      # dL/dz
        Gh = np.matmul(D.T[None], Gz)                      # dL/dh  [e, R, C]
        Gu = g[:, :, None] * Gh                            # dL/du
        np.add.at(grad_x, src[ids], np.matmul(A[None], Gu))
        dg = np.sum(Gh * u, axis=2)                        # dL/dg  [e, R]
        dv = dg * rho
        drho = dg * v
        grad_wrad += phi.T @ drho                          # [n, R]
        dY = dv @ B.T                                      # [e, d]
        dphi_w = drho @ Wrad.T                             # dL/dphi [e, n]
        J = spherical_harmonics_jacobian(L, vec)           # [e, d, 3]
        gv = np.einsum("ek,ekx->ex", dY, J)
        gv += (np.sum(dphi_w * dphi, axis=1) / dist)[:, None] * vec
        grad_vec[ids] = gv
    if return_radial:
        return grad_x, grad_W, grad_vec, grad_wrad
    return grad_x, grad_W, grad_vec


# ----------------------------------------------------------------- sampling
def forward_at_nodes(nodes, x, edge_index, edge_vec, A, B, D, W, radial_w, r_cut, L):
    """out[nodes] only, from the edges into those nodes (in sorted order)."""
    nodes = np.asarray(nodes, np.int64)
    dst = np.asarray(edge_index[1], np.int64)
    N = x.shape[0]
    perm, _ = stable_sort_by_key(dst, N)
    keep = np.zeros(N, bool)
    keep[nodes] = True
    sub = perm[keep[dst[perm]]]
    out = forward(x, edge_index, edge_vec, A, B, D, W, radial_w, r_cut, L, perm=sub)
    return out[nodes]
