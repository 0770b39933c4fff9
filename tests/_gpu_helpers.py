"""Shared helpers for the GPU parity tests: cached workloads and factor
fixtures, device upload, and the error metrics used for parity.

Parity metrics:
* rel_err: the relative Frobenius error ||gpu - oracle|| / ||oracle|| per
  output tensor, at most 1e-5 for float32 inputs and 2e-2 for bfloat16
  inputs, and no non-finite values;
* check_rows: the same bound per row of a tensor whose leading index is a
  node (or an edge), plus an elementwise bound |gpu - oracle| <= tol times the
  row's largest |oracle| value; rows whose oracle value is exactly zero (nodes
  without edges) must be exactly zero on the GPU;
* check_elementwise: |gpu - oracle| <= tol times the largest |oracle| value
  of the whole tensor (for the channel-by-channel grad_W and the radial-weight
  gradient, which have no node rows);
* check_scaled: per edge of grad_edge_vec, |gpu - oracle| <= tol times
  max(|oracle edge|, s_e / c), with s_e the edge's magnitude scale
  (grad_vec_scale: the same chain of products and sums evaluated on absolute
  values) and c the median of s_e / |oracle edge| over the edges.  An
  edge's gradient is a sum of terms of both signs (over channels, ranks,
  degree rows and radial functions) that can cancel to far below the terms;
  no floating-point evaluation keeps a small relative error there (a plain
  float32 evaluation of the oracle's own chain reaches 1e-5 per edge), while
  its error stays proportional to s_e.  So an edge of typical conditioning is
  held to its own relative error, and an edge conditioned k times worse than
  the median to k times that."""
from __future__ import annotations

import functools
import os

import numpy as np
import torch

import workloads

HERE = os.path.dirname(os.path.abspath(__file__))
FACTORS = os.path.join(HERE, "golden", "factors")
TOL_F32 = 1e-5
TOL_BF16 = 2e-2


def load_factors(L: int, R: int):
    z = np.load(os.path.join(FACTORS, f"cp_L{L}_R{R}.npz"))
    return z["A"], z["B"], z["D"]


@functools.lru_cache(maxsize=None)
def workload(name: str) -> dict:
    return workloads.make_workload(name)


def random_factors(L: int, R: int, seed: int):
    rng = np.random.default_rng(seed)
    d = (L + 1) ** 2
    return tuple((rng.standard_normal((d, R)) / np.sqrt(d)).astype(np.float32) for _ in range(3))


def device_inputs(w: dict, A, B, D, dev="cuda"):
    bf16 = w["feat_dtype"] == "bf16"
    t = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dev, dt)  # noqa: E731
    if bf16:
        x = torch.from_numpy(w["x_bf16"].view(np.int16)).to(dev).view(torch.bfloat16)
        W = torch.from_numpy(w["W_bf16"].view(np.int16)).to(dev).view(torch.bfloat16)
    else:
        x, W = t(w["x"]), t(w["W"])
    return dict(x=x, edge_vec=t(w["edge_vec"]), edge_index=torch.from_numpy(w["edge_index"]).to(dev),
                A=t(A), B=t(B), D=t(D), W=W, radial_w=t(w["radial_w"]))


def rel_err(gpu, ref) -> float:
    """Relative Frobenius error; with TDN_PARITY_LOG set, each value is also
    appended to that file with the running test's id."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert np.all(np.isfinite(gpu)), "non-finite values in GPU output"
    nrm = np.linalg.norm(ref)
    err = float(np.linalg.norm(gpu - ref) / (nrm if nrm > 0 else 1.0))
    log = os.environ.get("TDN_PARITY_LOG")
    if log:
        test = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
        with open(log, "a") as f:
            f.write(f"{test}\t{gpu.shape}\t{err:.3e}\n")
    return err


def _log(kind: str, shape, err: float):
    log = os.environ.get("TDN_PARITY_LOG")
    if log:
        test = os.environ.get("PYTEST_CURRENT_TEST", "?").split(" ")[0]
        with open(log, "a") as f:
            f.write(f"{test}\t{kind}\t{shape}\t{err:.3e}\n")


def check_rows(gpu, ref, tol: float, what: str = "") -> tuple[float, float]:
    """Per-row bounds (rows = leading index).  Returns the worst per-row
    relative Frobenius error and the worst elementwise error relative to its
    row's largest reference magnitude; asserts both are <= tol."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (what, gpu.shape, ref.shape)
    n = gpu.shape[0]
    if n == 0:
        return 0.0, 0.0
    g2, r2 = gpu.reshape(n, -1), ref.reshape(n, -1)
    assert np.all(np.isfinite(g2)), f"{what}: non-finite values in GPU output"
    rnorm = np.linalg.norm(r2, axis=1)
    rmax = np.max(np.abs(r2), axis=1)
    zero = rnorm == 0
    assert np.all(g2[zero] == 0), f"{what}: nonzero GPU values in rows whose reference is zero"
    nz = ~zero
    if not np.any(nz):
        return 0.0, 0.0
    diff = g2[nz] - r2[nz]
    rel = np.linalg.norm(diff, axis=1) / rnorm[nz]
    elem = np.max(np.abs(diff), axis=1) / rmax[nz]
    worst_rel, worst_elem = float(rel.max()), float(elem.max())
    _log("rows_rel", gpu.shape, worst_rel)
    _log("rows_elem", gpu.shape, worst_elem)
    assert worst_rel <= tol, f"{what}: worst row relative error {worst_rel:.3e} (row {int(np.argmax(rel))})"
    assert worst_elem <= tol, f"{what}: worst elementwise error {worst_elem:.3e} of its row's max"
    return worst_rel, worst_elem


def check_elementwise(gpu, ref, tol: float, what: str = "") -> float:
    """|gpu - ref| <= tol max|ref| over the whole tensor; returns the ratio."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite values in GPU output"
    m = float(np.max(np.abs(ref))) if ref.size else 0.0
    err = float(np.max(np.abs(gpu - ref))) / (m if m > 0 else 1.0) if ref.size else 0.0
    _log("elem", gpu.shape, err)
    assert err <= tol, f"{what}: elementwise error {err:.3e} of the tensor's max"
    return err


def grad_vec_scale(w: dict, A, B, D, G=None, edges=None) -> np.ndarray:
    """Per-edge magnitude scale [len(edges), 3] of dL/dr_e: the chain
    dg = sum_c (D^T G W^T)[t] * (A^T x[s]), dY = B (dg * rho),
    dphi = Wrad (dg * v), dL/dr = J^T dY + (sum_q dphi_q phi'_q) r/|r|
    with every factor, harmonic, Jacobian entry and radial value replaced by
    its absolute value (an error-bound scale, not a reference value)."""
    from oracle import layer, sh

    x = np.abs(np.asarray(w["x"], np.float64))
    G = np.abs(np.asarray(w["grad_out"] if G is None else G, np.float64))
    Wa = np.abs(np.asarray(w["W"], np.float64))
    Aa, Ba, Da = (np.abs(np.asarray(m, np.float64)) for m in (A, B, D))
    Wr = np.abs(np.asarray(w["radial_w"], np.float64))
    src, dst = np.asarray(w["edge_index"], np.int64)
    edges = np.arange(w["E"]) if edges is None else np.asarray(edges, np.int64)
    out = np.zeros((edges.shape[0], 3))
    for c0 in range(0, edges.shape[0], 256):
        ids = edges[c0:c0 + 256]
        vec = np.asarray(w["edge_vec"], np.float64)[ids]
        dist = np.linalg.norm(vec, axis=1)
        Y = np.abs(sh.spherical_harmonics(w["L"], vec))
        J = np.abs(sh.spherical_harmonics_jacobian(w["L"], vec))
        phi, dphi = layer.radial_basis(dist, w["r_cut"], Wr.shape[0])
        phi, dphi = np.abs(phi), np.abs(dphi)
        u = np.matmul(Aa.T[None], x[src[ids]])
        Gh = np.matmul(Da.T[None], G[dst[ids]] @ Wa.T)
        dg = np.sum(Gh * u, axis=2)
        v, rho = Y @ Ba, phi @ Wr
        dY = (dg * rho) @ Ba.T
        dphi_w = (dg * v) @ Wr.T
        out[c0:c0 + ids.shape[0]] = (np.einsum("ek,ekx->ex", dY, J)
                                     + (np.sum(dphi_w * dphi, axis=1) / dist)[:, None] * np.abs(vec))
    return out


def check_scaled(gpu, ref, scale, tol: float, what: str = "") -> float:
    """The per-edge bound described above; returns the worst ratio of the
    error to its bound."""
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    scale = np.asarray(scale, np.float64)
    assert np.all(np.isfinite(gpu)), f"{what}: non-finite values in GPU output"
    n = gpu.shape[0]
    if n == 0:
        return 0.0
    d = np.max(np.abs(gpu - ref).reshape(n, -1), axis=1)
    r = np.max(np.abs(ref).reshape(n, -1), axis=1)
    s = np.max(scale.reshape(n, -1), axis=1)
    assert np.all(s >= r * (1 - 1e-9)), f"{what}: magnitude scale below the value it bounds"
    assert np.all(d[s == 0] == 0), f"{what}: nonzero error where the scale is zero"
    ok = r > 0
    if not np.any(ok):
        return 0.0
    c = float(np.median(s[ok] / r[ok]))
    bound = np.maximum(r, s / c)
    pos = bound > 0
    ratio = d[pos] / bound[pos]
    err = float(ratio.max()) if ratio.size else 0.0
    _log("scaled", gpu.shape, err)
    assert err <= tol, f"{what}: error {err:.3e} of its conditioning-adjusted magnitude"
    return err


def tol(w: dict) -> float:
    return TOL_BF16 if w["feat_dtype"] == "bf16" else TOL_F32


def sample_nodes(w: dict, k: int, seed: int = 0, by: int = 1) -> np.ndarray:
    """k seeded nodes plus the first, the last and the one of largest degree
    (by=1: in-degree, by=0: out-degree)."""
    N = w["N"]
    rng = np.random.default_rng(seed)
    deg = np.bincount(w["edge_index"][by], minlength=N)
    extra = [0, N - 1, int(np.argmax(deg))]
    return np.unique(np.concatenate([rng.choice(N, size=min(k, N), replace=False), extra]))
