"""The attention block that consumes the CP messages -- TEST INFRASTRUCTURE
ONLY (only tests/, the smoke check and the benchmark's CPU leg use it).

Sec. 4.1 ("Model Design") builds TDN on Equiformer's graph transformer: its
graph attention (MLP attention) keeps its structure and the CG tensor products
inside it become the rank-R CP product with path-weight sharing (Sec. 3.1,
Sec. 3.2).  The paper gives no equations for the block, so this module fixes
one reading of it, the one the GPU path implements:

    messages  z_e = D diag(g_e) A^T x[s_e]            [d, C], the layer's CP
              product for edge e = (s, t) before the channel weight W
    logits    q_e = [x[t]^(0), x[s]^(0), phi_e]       invariant inputs: the
              degree-0 rows of both nodes and the radial basis of |r_e|
              a_e = LeakyReLU(q_e W1; 0.2) w2         [H], one per head
    weights   alpha_e[h] = exp(a_e[h]) / sum over e' into t of exp(a_e'[h])
    output    out[t][:, c] = sum over e into t of alpha_e[c // (C/H)] z_e[:, c],
              then out[t] W

Heads split the C channels into H contiguous groups.  Everything is float64
and per edge (D per edge, nothing reassociated); the largest logit of each
destination and head is subtracted before exp, which changes no value.
"""
from __future__ import annotations

import numpy as np

from .layer import edge_terms, radial_basis, stable_sort_by_key

LEAKY_SLOPE = 0.2


def leaky_relu(v, slope=LEAKY_SLOPE):
    return np.where(v > 0, v, slope * v)


def logits(x, edge_index, edge_vec, W1, w2, r_cut, n_radial):
    """a [E, H] by edge id."""
    x = np.asarray(x, np.float64)
    src = np.asarray(edge_index[0], np.int64)
    dst = np.asarray(edge_index[1], np.int64)
    vec = np.asarray(edge_vec, np.float64)
    phi, _ = radial_basis(np.linalg.norm(vec, axis=1), r_cut, n_radial)
    q = np.concatenate([x[dst, 0, :], x[src, 0, :], phi], axis=1)      # [E, 2C + n_radial]
    return leaky_relu(q @ np.asarray(W1, np.float64)) @ np.asarray(w2, np.float64)


def segment_softmax(a, dst, n_nodes):
    """alpha [E, H]: a softmax over the edges of each destination, per head."""
    a = np.asarray(a, np.float64)
    dst = np.asarray(dst, np.int64)
    mx = np.full((n_nodes, a.shape[1]), -np.inf)
    np.maximum.at(mx, dst, a)
    ex = np.exp(a - mx[dst])
    den = np.zeros((n_nodes, a.shape[1]))
    np.add.at(den, dst, ex)
    return ex / den[dst]


def forward(x, edge_index, edge_vec, A, B, D, W, radial_w, W1, w2, r_cut, L, perm=None, return_z=False):
    """(out [N, d, C], alpha [E, H] by edge id), and the weighted sum before W
    with return_z."""
    x = np.asarray(x, np.float64)
    A, B, D, W = (np.asarray(v, np.float64) for v in (A, B, D, W))
    N, d, C = x.shape
    H = np.asarray(w2).shape[1]
    assert C % H == 0
    src = np.asarray(edge_index[0], np.int64)
    dst = np.asarray(edge_index[1], np.int64)
    alpha = segment_softmax(logits(x, edge_index, edge_vec, W1, w2, r_cut, np.asarray(radial_w).shape[0]), dst, N)
    if perm is None:
        perm, _ = stable_sort_by_key(dst, N)
    perm = np.asarray(perm, np.int64)
    head = np.arange(C) // (C // H)
    zsum = np.zeros((N, d, C))
    for e in perm:                                                 # in sorted order
        _, _, _, _, g = edge_terms(np.asarray(edge_vec)[e:e + 1], L, B, radial_w, r_cut)
        z = D @ (g[0][:, None] * (A.T @ x[src[e]]))                # [d, C]
        zsum[dst[e]] += alpha[e][head][None, :] * z
    out = zsum @ W
    return (out, alpha, zsum) if return_z else (out, alpha)
