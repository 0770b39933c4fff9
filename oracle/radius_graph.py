"""Radius graph of a batch of atomic systems by brute force -- TEST
INFRASTRUCTURE ONLY (see the package header).

The layer's edges come from a radius graph built on the fly (App. "Model and
Training Configurations": cutoff 5.0 with at most 500 neighbours for OC20,
cutoff 12.0 with at most 20 for OC22).  Definition used here:

* A batch holds G independent systems; system g owns the atoms
  graph_ptr[g] .. graph_ptr[g+1]-1 and, on each periodic axis a, a box of
  length cell[g, a] with the atoms' coordinates in [0, cell[g, a]).
* A directed edge (src, dst, n) joins two atoms of the same system through
  the source image n (an integer per axis, zero on non-periodic axes):
      r = (pos[src] - pos[dst]) + n * cell[g]
  is the edge vector, and the edge exists when |r|^2 < r_cut^2, except the
  atom itself (src == dst with n = 0).  Boxes are at least r_cut long on
  every periodic axis, so only n in {-1, 0, 1} can qualify.
* Decisions and vectors are float32: the difference of the float32
  positions, then the image added, each rounded; |r|^2 as
  ((rx*rx + ry*ry) + rz*rz) with every product and sum rounded to float32
  (no fused multiply-add), compared with the float32 product r_cut*r_cut.
  The paper does not fix a precision; float32 is the precision of the edge
  vectors the layer consumes.
* With a neighbour cap K > 0 each destination keeps the K candidates
  smallest in (|r|^2, src, image code); without one it keeps all.
* Order: by destination, then source, then image code
  (nx+1)*9 + (ny+1)*3 + (nz+1).

Every atom pair of every system is tested against every image, in plain
numpy: slow, and obviously the definition above.
"""
from __future__ import annotations

import itertools

import numpy as np

f32 = np.float32


def image_code(n) -> np.ndarray:
    n = np.asarray(n, dtype=np.int64)
    return (n[..., 0] + 1) * 9 + (n[..., 1] + 1) * 3 + (n[..., 2] + 1)


def _images(periodic):
    axes = [(-1, 0, 1) if p else (0,) for p in periodic]
    return np.array(list(itertools.product(*axes)), dtype=np.int64)


def _check(pos, graph_ptr, cell, periodic, r_cut):
    pos = np.asarray(pos)
    assert pos.dtype == np.float32 and pos.ndim == 2 and pos.shape[1] == 3
    ptr = np.asarray(graph_ptr, dtype=np.int64)
    assert ptr[0] == 0 and ptr[-1] == pos.shape[0] and np.all(np.diff(ptr) >= 0)
    per = tuple(bool(p) for p in periodic)
    if any(per):
        cell = np.asarray(cell, dtype=np.float32).reshape(len(ptr) - 1, 3)
        for g in range(len(ptr) - 1):
            for a in range(3):
                if per[a]:
                    assert cell[g, a] >= f32(r_cut), "box shorter than the cutoff"
                    x = pos[ptr[g]:ptr[g + 1], a]
                    assert np.all((x >= 0) & (x < cell[g, a])), "coordinate outside [0, L)"
    else:
        cell = np.zeros((len(ptr) - 1, 3), dtype=np.float32)
    return pos, ptr, cell, per


def radius_graph(pos, graph_ptr, cell, periodic, r_cut, max_neighbors=0, dst_nodes=None):
    """Edges of the definition above.

    pos float32 [N,3]; graph_ptr [G+1]; cell float32 [G,3] (used on periodic
    axes only; may be None when no axis is periodic); periodic 3 bools;
    r_cut; max_neighbors (0 = no cap); dst_nodes: optional subset of
    destination atoms (default all).

    Returns (src int64 [E], dst int64 [E], image int64 [E,3],
    vec float32 [E,3]) in (dst, src, image code) order."""
    pos, ptr, cell, per = _check(pos, graph_ptr, cell, periodic, r_cut)
    N = pos.shape[0]
    rc2 = f32(r_cut) * f32(r_cut)
    imgs = _images(per)                                    # [I, 3]
    graph_of = np.repeat(np.arange(len(ptr) - 1), np.diff(ptr))
    dsts = np.arange(N) if dst_nodes is None else np.asarray(dst_nodes, dtype=np.int64)
    out_s, out_d, out_n, out_v = [], [], [], []
    for d in dsts:
        g = graph_of[d]
        a, b = ptr[g], ptr[g + 1]
        src = np.arange(a, b)
        t = pos[a:b] - pos[d]                              # float32 [m, 3]
        shift = (imgs.astype(np.float32) * cell[g])        # [I, 3], entries 0 or +-L exactly
        r = t[:, None, :] + shift[None, :, :]              # float32 [m, I, 3]
        r2 = (r[..., 0] * r[..., 0] + r[..., 1] * r[..., 1]) + r[..., 2] * r[..., 2]
        ok = r2 < rc2
        ok[d - a, np.all(imgs == 0, axis=1)] = False
        si, ii = np.nonzero(ok)
        s_e, n_e, v_e, r2_e = src[si], imgs[ii], r[si, ii], r2[si, ii]
        code = image_code(n_e)
        if max_neighbors and s_e.shape[0] > max_neighbors:
            keep = np.lexsort((code, s_e, r2_e))[:max_neighbors]
            s_e, n_e, v_e, code = s_e[keep], n_e[keep], v_e[keep], code[keep]
        o = np.lexsort((code, s_e))
        out_s.append(s_e[o])
        out_d.append(np.full(o.shape[0], d, dtype=np.int64))
        out_n.append(n_e[o])
        out_v.append(v_e[o])
    if not out_s:
        return (np.zeros(0, np.int64), np.zeros(0, np.int64), np.zeros((0, 3), np.int64),
                np.zeros((0, 3), np.float32))
    return (np.concatenate(out_s), np.concatenate(out_d), np.concatenate(out_n).reshape(-1, 3),
            np.concatenate(out_v).reshape(-1, 3).astype(np.float32))

