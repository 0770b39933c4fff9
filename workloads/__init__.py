"""Seeded synthetic workloads for the CP tensor-product message-passing layer.

This package is shared by the oracle tests and the GPU path, so it holds none
of the layer's arithmetic: it only draws atom positions, radius graphs, node
features, the channel-mix weight W, the radial weight matrix and the output
cotangent, each from its own seeded stream.  The CP factors are not drawn
here: they are fitted once, offline, to the Clebsch-Gordan tensor and cached
as files (the paper precomputes and caches the factors per maximum degree,
Sec. 4.1 "Model Design").

Five workloads are defined; each is named by what it is and its sizes.  The
headline one is ``molecules3200_L4_C128_R128``.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from . import geometry

N_RADIAL = 8


@dataclass(frozen=True)
class Workload:
    name: str
    L: int
    C: int
    R: int
    r_cut: float
    feat_dtype: str          # "f32" or "bf16": dtype of x and W; everything else is f32
    presorted: bool          # edges emitted sorted by (dst, src)
    backward: bool           # workload exercises the backward pass
    seed: int

    @property
    def d(self) -> int:
        return (self.L + 1) ** 2


WORKLOADS = {
    w.name: w
    for w in [
        Workload("cube64_L2_C16_R32", 2, 16, 32, 3.0, "f32", True, False, 1000),
        Workload("molecules960_L3_C64_R64", 3, 64, 64, 5.0, "f32", True, True, 1001),
        Workload("molecules3200_L4_C128_R128", 4, 128, 128, 6.0, "f32", True, False, 1002),
        Workload("slabs4960_L6_C128_R256", 6, 128, 256, 6.0, "f32", True, True, 1003),
        Workload("bulk4096_L4_C256_R128_bf16", 4, 256, 128, 6.0, "bf16", False, True, 1004),
    ]
}
HEADLINE = "molecules3200_L4_C128_R128"


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even).

    Returns the bf16 bit patterns as uint16."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    bits = a.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = (bits + 0x7FFF + lsb) >> 16
    nan = np.isnan(a)
    out = rounded.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def _streams(seed: int):
    names = ["pos", "x", "W", "Wrad", "grad", "perm", "spare1", "spare2"]
    kids = np.random.SeedSequence(seed).spawn(len(names))
    return {n: np.random.default_rng(k) for n, k in zip(names, kids)}


def _batch_of_molecules(rng, n_graphs, n_atoms, sphere):
    return [geometry.molecule_walk(rng, n_atoms, sphere=sphere, ring_start=bool(g % 2)) for g in range(n_graphs)]


def _slabs(rng, n_slabs):
    graphs, cells = [], []
    for _ in range(n_slabs):
        slab, cell_xy = geometry.fcc_slab(rng)
        ads = geometry.molecule_walk(rng, 10, sphere=3.0)
        top = slab[:, 2].max()
        shift = np.array([rng.uniform(0, cell_xy[0]), rng.uniform(0, cell_xy[1]),
                          top + 2.0 - ads[:, 2].min()])
        ads = ads - ads[0] * np.array([1.0, 1.0, 0.0]) + shift
        ads[:, :2] %= cell_xy
        graphs.append(np.concatenate([slab, ads]))
        cells.append(np.array([cell_xy[0], cell_xy[1], 0.0]))
    return graphs, cells


def make_geometry(w: Workload) -> dict:
    """The atoms behind a workload's graph: a batch of independent graphs.

    Returns pos float64 [N,3] (graphs one after another), graph_ptr int64
    [G+1] (graph g holds atoms graph_ptr[g] .. graph_ptr[g+1]-1), cell
    float64 [G,3] (box lengths; 0 on non-periodic axes), periodic (3 bools)
    and r_cut.  Periodic coordinates are as generated (slab atoms may lie up
    to a few tenths of an Angstrom outside [0, L))."""
    rng = _streams(w.seed)["pos"]
    if w.name.startswith("cube64"):
        graphs, cells, per = [rng.uniform(0.0, 6.0, size=(64, 3))], [np.zeros(3)], (False, False, False)
    elif w.name.startswith("molecules960"):
        graphs = _batch_of_molecules(rng, 32, 30, sphere=3.5)
        cells, per = [np.zeros(3)] * 32, (False, False, False)
    elif w.name.startswith("molecules3200"):
        graphs = _batch_of_molecules(rng, 64, 50, sphere=3.5)
        cells, per = [np.zeros(3)] * 64, (False, False, False)
    elif w.name.startswith("slabs4960"):
        graphs, cells = _slabs(rng, 16)
        per = (True, True, False)
    elif w.name.startswith("bulk4096"):
        box = (4096 / 0.1) ** (1.0 / 3.0)
        graphs = [geometry.random_sequential_addition(rng, 4096, box)]
        cells, per = [np.array([box, box, box])], (True, True, True)
    else:
        raise KeyError(w.name)
    ptr = np.concatenate([[0], np.cumsum([g.shape[0] for g in graphs])]).astype(np.int64)
    return dict(pos=np.concatenate(graphs), graph_ptr=ptr, cell=np.stack(cells), periodic=per, r_cut=float(w.r_cut))


def graph_inputs(name: str) -> dict:
    """A workload's geometry as the radius-graph builder takes it: float32
    positions wrapped into [0, L) on periodic axes (a coordinate that rounds
    up to L becomes 0), int32 graph_ptr, float32 cell, periodic, r_cut."""
    g = make_geometry(WORKLOADS[name])
    return wrap_inputs(g["pos"], g["graph_ptr"], g["cell"], g["periodic"], g["r_cut"])


def wrap_inputs(pos, graph_ptr, cell, periodic, r_cut) -> dict:
    ptr = np.asarray(graph_ptr, dtype=np.int64)
    cell = np.asarray(cell, dtype=np.float64).reshape(len(ptr) - 1, 3)
    p = np.array(pos, dtype=np.float64)
    for k in range(len(ptr) - 1):
        for a in range(3):
            if periodic[a]:
                p[ptr[k]:ptr[k + 1], a] = np.mod(p[ptr[k]:ptr[k + 1], a], cell[k, a])
    p32 = p.astype(np.float32)
    cell32 = cell.astype(np.float32)
    for k in range(len(ptr) - 1):
        for a in range(3):
            if periodic[a]:
                col = p32[ptr[k]:ptr[k + 1], a]
                col[col >= cell32[k, a]] = 0.0
    return dict(pos=p32, graph_ptr=ptr.astype(np.int32), cell=cell32, periodic=tuple(bool(x) for x in periodic),
                r_cut=float(r_cut))


def make_graph(w: Workload):
    """Returns (n_nodes, src, dst, edge_vec) for a workload (float64 vectors):
    the radius graph of every graph of ``make_geometry``, concatenated."""
    g = make_geometry(w)
    pos, ptr, per = g["pos"], g["graph_ptr"], g["periodic"]
    srcs, dsts, vecs = [], [], []
    for k in range(len(ptr) - 1):
        a, b = int(ptr[k]), int(ptr[k + 1])
        if any(per):
            s, t, v = geometry.radius_graph(pos[a:b], g["r_cut"], g["cell"][k], per)
        else:
            s, t, v = geometry.radius_graph(pos[a:b], g["r_cut"])
        srcs.append(s + a)
        dsts.append(t + a)
        vecs.append(v)
    return int(ptr[-1]), np.concatenate(srcs), np.concatenate(dsts), np.concatenate(vecs)


def make_workload(name: str) -> dict:
    """Draws every input of one workload.

    Returns a dict with
      N, E, L, d, C, R, r_cut, n_radial, feat_dtype, presorted
      edge_index int32 [2,E] (row 0 = src, row 1 = dst), in the order handed
                 to the layer (sorted by (dst, src) when ``presorted``,
                 otherwise a seeded random permutation of that order)
      edge_vec   float32 [E,3]
      x          float32 [N,d,C]  (values exactly representable in bf16 when
                 feat_dtype == "bf16"; ``x_bf16`` then holds the bit patterns)
      W          float32 [C,C]    (likewise ``W_bf16``)
      radial_w   float32 [n_radial,R]
      grad_out   float32 [N,d,C]
    """
    w = WORKLOADS[name]
    st = _streams(w.seed)
    n, src, dst, vec = make_graph(w)
    if not w.presorted:
        p = st["perm"].permutation(src.shape[0])
        src, dst, vec = src[p], dst[p], vec[p]
    d, C, R = w.d, w.C, w.R
    x = st["x"].standard_normal((n, d, C), dtype=np.float32)
    W = (st["W"].standard_normal((C, C)) / np.sqrt(C)).astype(np.float32)
    radial_w = (st["Wrad"].standard_normal((N_RADIAL, R)) / np.sqrt(N_RADIAL)).astype(np.float32)
    grad_out = st["grad"].standard_normal((n, d, C), dtype=np.float32)
    out = dict(name=name, N=int(n), E=int(src.shape[0]), L=w.L, d=d, C=C, R=R,
               r_cut=float(w.r_cut), n_radial=N_RADIAL, feat_dtype=w.feat_dtype,
               presorted=w.presorted, backward=w.backward,
               edge_index=np.stack([src, dst]).astype(np.int32),
               edge_vec=vec.astype(np.float32), radial_w=radial_w, grad_out=grad_out)
    if w.feat_dtype == "bf16":
        out["x_bf16"] = bf16_round(x)
        out["W_bf16"] = bf16_round(W)
        out["x"] = bf16_to_f32(out["x_bf16"])
        out["W"] = bf16_to_f32(out["W_bf16"])
    else:
        out["x"] = x
        out["W"] = W
    return out


def random_graph(seed: int, n_nodes: int, n_edges: int, L: int, C: int, R: int,
                 r_cut: float = 5.0, sort: bool = False, feat_dtype: str = "f32") -> dict:
    """A small seeded random graph for edge cases (ragged segments, isolated
    nodes, skewed degrees).  Edge vectors are random with lengths in
    [0.3, r_cut); duplicate (src, dst) pairs are allowed."""
    st = _streams(seed)
    rng = st["pos"]
    src = rng.integers(0, max(n_nodes, 1), size=n_edges)
    dst = rng.integers(0, max(n_nodes, 1), size=n_edges)
    u = rng.normal(size=(n_edges, 3))
    u /= np.linalg.norm(u, axis=1, keepdims=True)
    vec = u * rng.uniform(0.3, r_cut, size=(n_edges, 1))
    if sort:
        o = np.lexsort((src, dst))
        src, dst, vec = src[o], dst[o], vec[o]
    d = (L + 1) ** 2
    x = st["x"].standard_normal((n_nodes, d, C), dtype=np.float32)
    W = (st["W"].standard_normal((C, C)) / np.sqrt(max(C, 1))).astype(np.float32)
    radial_w = (st["Wrad"].standard_normal((N_RADIAL, R)) / np.sqrt(N_RADIAL)).astype(np.float32)
    grad_out = st["grad"].standard_normal((n_nodes, d, C), dtype=np.float32)
    out = dict(name=f"random_{seed}", N=n_nodes, E=n_edges, L=L, d=d, C=C, R=R,
               r_cut=float(r_cut), n_radial=N_RADIAL, feat_dtype=feat_dtype, presorted=sort,
               backward=True, edge_index=np.stack([src, dst]).astype(np.int32),
               edge_vec=vec.astype(np.float32), radial_w=radial_w, grad_out=grad_out)
    if feat_dtype == "bf16":
        out["x_bf16"] = bf16_round(x)
        out["W_bf16"] = bf16_round(W)
        out["x"] = bf16_to_f32(out["x_bf16"])
        out["W"] = bf16_to_f32(out["W_bf16"])
    else:
        out["x"], out["W"] = x, W
    return out
