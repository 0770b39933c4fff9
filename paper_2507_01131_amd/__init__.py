"""MI355X (gfx950) CP tensor-product message-passing layer of Tensor
Decomposition Networks (arXiv 2507.01131).

This module is the Python binding of ``libtdn.so`` (ctypes).  It only
marshals arguments: every step of the layer runs in the library's HIP
kernels; torch provides device memory and the current stream.  It raises if
the library is not built -- there is no fallback implementation.

    import paper_2507_01131_amd as tdn
    res = tdn.forward(x, edge_vec, edge_index, A, B, D, W, radial_w, L=4, r_cut=6.0)
    grads = tdn.backward(res, grad_out)
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

__all__ = ["forward", "backward", "sort_by_key", "spherical_harmonics", "workspace_size", "Problem",
           "TdnError", "lib", "timer_enable", "timer_read", "LIB_PATH", "status_string"]

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libtdn.so")

TDN_F32, TDN_BF16 = 0, 1
STATUS = {0: "TDN_OK", 1: "TDN_ERR_NULL_POINTER", 2: "TDN_ERR_BAD_SHAPE", 3: "TDN_ERR_BAD_DTYPE",
          4: "TDN_ERR_WORKSPACE_TOO_SMALL", 5: "TDN_ERR_INDEX_OUT_OF_RANGE", 6: "TDN_ERR_NOT_SORTED",
          7: "TDN_ERR_DEGENERATE_EDGE", 8: "TDN_ERR_UNSUPPORTED_DEVICE", 9: "TDN_ERR_HIP",
          10: "TDN_ERR_BAD_GEOMETRY", 11: "TDN_ERR_EDGE_CAPACITY", 12: "TDN_ERR_NEIGHBOUR_LIMIT",
          13: "TDN_ERR_SCRATCH_LIMIT"}
TDN_ERR_EDGE_CAPACITY = 11


class TdnError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        extra = ""
        if status == 9:
            extra = f" (hipError {lib().tdn_last_hip_error()})"
        super().__init__(f"{where}: {STATUS.get(status, status)}{extra}")


class GraphProblem(ctypes.Structure):
    _fields_ = [("n_nodes", ctypes.c_int32), ("n_graphs", ctypes.c_int32), ("r_cut", ctypes.c_float),
                ("max_neighbors", ctypes.c_int32), ("periodic", ctypes.c_int32 * 3)]


class Problem(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("C", ctypes.c_int32), ("R", ctypes.c_int32),
                ("n_nodes", ctypes.c_int32), ("n_edges", ctypes.c_int32), ("n_radial", ctypes.c_int32),
                ("r_cut", ctypes.c_float), ("feat_dtype", ctypes.c_int32), ("edges_sorted", ctypes.c_int32),
                ("validate", ctypes.c_int32)]


_lib = None
_P = ctypes.c_void_p
_SZ = ctypes.c_size_t


def lib() -> ctypes.CDLL:
    """The loaded libtdn.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_2507_01131_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        PP = ctypes.POINTER(Problem)
        L.tdn_workspace_size.argtypes = [PP, ctypes.POINTER(_SZ), ctypes.POINTER(_SZ)]
        L.tdn_cp_tp_forward.argtypes = [PP] + [_P] * 13 + [_SZ, _P]
        L.tdn_ablation_forward_atomics.argtypes = [PP] + [_P] * 13 + [_SZ, _P]
        L.tdn_cp_tp_forward_noalloc.argtypes = [PP] + [_P] * 13
        L.tdn_cp_tp_backward.argtypes = [PP] + [_P] * 17 + [_SZ, _P]
        L.tdn_ps_linear_workspace_size.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(_SZ)]
        L.tdn_ps_linear.argtypes = [ctypes.c_int32] * 3 + [_P, _P, ctypes.c_int32, _P, _P, _SZ, _P]
        L.tdn_cp_tp3_forward.argtypes = [PP] + [_P] * 14 + [_SZ, _P]
        L.tdn_dense_tp_forward.argtypes = [PP] + [_P] * 6 + [ctypes.c_int32] + [_P] * 7 + [_SZ, _P]
        L.tdn_dense_tp_unshared_workspace_size.argtypes = [PP, ctypes.POINTER(_SZ)]
        L.tdn_ablation_workspace_size.argtypes = [PP, ctypes.c_int32, ctypes.POINTER(_SZ)]
        L.tdn_attention_workspace_size.argtypes = [PP, ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(_SZ)]
        L.tdn_attention_forward.argtypes = [PP, ctypes.c_int32, ctypes.c_int32] + [_P] * 16 + [_SZ, _P]
        L.tdn_ablation_forward.argtypes = [PP, ctypes.c_int32] + [_P] * 13 + [_SZ, _P]
        L.tdn_dense_tp_forward_unshared.argtypes = [PP] + [_P] * 6 + [ctypes.c_int32] + [_P] * 6 + [_SZ, _P]
        GP = ctypes.POINTER(GraphProblem)
        L.tdn_radius_graph_workspace_size.argtypes = [GP, ctypes.POINTER(_SZ)]
        L.tdn_radius_graph.argtypes = [GP, _P, _P, _P, ctypes.c_int64, _P, _P, _P, _P,
                                       ctypes.POINTER(ctypes.c_int64), _P, _SZ, _P]
        L.tdn_sort_workspace_size.argtypes = [ctypes.c_int32, ctypes.c_int32, ctypes.POINTER(_SZ)]
        L.tdn_sort_by_key.argtypes = [ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P, _SZ, _P]
        L.tdn_spherical_harmonics.argtypes = [ctypes.c_int32, ctypes.c_int32, _P, _P, _P, _P]
        L.tdn_timer_enable.argtypes = [ctypes.c_int32]
        L.tdn_timer_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                     ctypes.POINTER(ctypes.c_int32), ctypes.c_int32]
        L.tdn_status_string.argtypes = [ctypes.c_int]
        L.tdn_status_string.restype = ctypes.c_char_p
        L.tdn_last_hip_error.restype = ctypes.c_int32
        for f in ("tdn_workspace_size", "tdn_cp_tp_forward", "tdn_ablation_forward_atomics", "tdn_cp_tp_backward",
                  "tdn_cp_tp_forward_noalloc",
                  "tdn_sort_workspace_size", "tdn_sort_by_key", "tdn_spherical_harmonics", "tdn_timer_enable",
                  "tdn_timer_read", "tdn_radius_graph_workspace_size", "tdn_radius_graph", "tdn_dense_tp_forward",
                  "tdn_cp_tp3_forward", "tdn_ps_linear_workspace_size", "tdn_ps_linear",
                  "tdn_dense_tp_unshared_workspace_size", "tdn_dense_tp_forward_unshared",
                  "tdn_ablation_workspace_size", "tdn_ablation_forward", "tdn_attention_workspace_size",
                  "tdn_attention_forward"):
            getattr(L, f).restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(s: int) -> str:
    return lib().tdn_status_string(s).decode()


def _check(status: int, where: str):
    if status != 0:
        raise TdnError(status, where)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def make_problem(L, C, R, n_nodes, n_edges, r_cut, n_radial=8, feat_dtype=TDN_F32, edges_sorted=False,
                 validate=False) -> Problem:
    return Problem(int(L), int(C), int(R), int(n_nodes), int(n_edges), int(n_radial), float(r_cut),
                   int(feat_dtype), int(bool(edges_sorted)), int(bool(validate)))


def workspace_size(p: Problem) -> tuple[int, int]:
    f, b = _SZ(), _SZ()
    _check(lib().tdn_workspace_size(ctypes.byref(p), ctypes.byref(f), ctypes.byref(b)), "tdn_workspace_size")
    return f.value, b.value


def _need(t, name, dtype, shape, device):
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name}: dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple(shape)}")
    if t.device != device:
        raise ValueError(f"{name}: on {t.device}, expected {device}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


@dataclass
class ForwardResult:
    out: torch.Tensor
    z: torch.Tensor | None
    perm: torch.Tensor
    offsets: torch.Tensor
    problem: Problem
    inputs: dict


def forward(x, edge_vec, edge_index, A, B, D, W, radial_w, *, L: int, r_cut: float, edges_sorted=False,
            validate=False, save_z=True, workspace=None, out=None, z=None, perm=None, offsets=None,
            stream=None, atomics_ablation=False, ablation=0) -> ForwardResult:
    """Runs tdn_cp_tp_forward.  x [N,d,C] and W [C,C] are float32 or bfloat16
    (both the same); edge_index [2,E] int32 (int64 is converted); everything
    else float32 on the same device.  out, z, perm, offsets and workspace may
    be passed preallocated; otherwise they are allocated here.
    atomics_ablation=True runs tdn_ablation_forward_atomics instead (the
    per-edge atomic scatter-add the segmented sum replaces; fp32, 2 <= L <= 4);
    ablation=ABL_FACTORS_GLOBAL, ABL_Y_TABLE or ABL_VALU runs
    tdn_ablation_forward with that variant."""
    dev = x.device
    N, d, C = x.shape
    E = edge_vec.shape[0]
    R = A.shape[1]
    if edge_index.dtype != torch.int32:
        edge_index = edge_index.to(torch.int32)
    edge_index = edge_index.contiguous()
    fd = TDN_BF16 if x.dtype == torch.bfloat16 else TDN_F32
    for t, n, dt, sh in [(x, "x", x.dtype, (N, d, C)), (edge_vec, "edge_vec", torch.float32, (E, 3)),
                         (edge_index, "edge_index", torch.int32, (2, E)), (A, "A", torch.float32, (d, R)),
                         (B, "B", torch.float32, (d, R)), (D, "D", torch.float32, (d, R)),
                         (W, "W", x.dtype, (C, C)), (radial_w, "radial_w", torch.float32, (radial_w.shape[0], R))]:
        _need(t, n, dt, sh, dev)
    if x.dtype not in (torch.float32, torch.bfloat16):
        raise TypeError("x must be float32 or bfloat16")
    p = make_problem(L, C, R, N, E, r_cut, radial_w.shape[0], fd, edges_sorted, validate)
    if ablation:
        fwd_bytes = ablation_workspace_size(p, ablation)
    else:
        fwd_bytes, _ = workspace_size(p)
    if workspace is None or workspace.numel() < fwd_bytes:
        workspace = torch.empty(max(fwd_bytes, 1), dtype=torch.uint8, device=dev)
    if out is None:
        out = torch.empty((N, d, C), dtype=torch.float32, device=dev)
    if z is None and save_z:
        z = torch.empty((N, d, C), dtype=torch.float32, device=dev)
    if perm is None:
        perm = torch.empty(max(E, 1), dtype=torch.int32, device=dev)[:E]
    if offsets is None:
        offsets = torch.empty(N + 1, dtype=torch.int32, device=dev)
    _need(out, "out", torch.float32, (N, d, C), dev)
    if z is not None:
        _need(z, "z", torch.float32, (N, d, C), dev)
    _need(perm, "perm", torch.int32, (E,), dev)
    _need(offsets, "offsets", torch.int32, (N + 1,), dev)
    if ablation:
        name = "tdn_ablation_forward"
        st = lib().tdn_ablation_forward(ctypes.byref(p), int(ablation), _ptr(x), _ptr(edge_vec), _ptr(edge_index),
                                        _ptr(A), _ptr(B), _ptr(D), _ptr(W), _ptr(radial_w), _ptr(out), _ptr(z),
                                        _ptr(perm), _ptr(offsets), _ptr(workspace), workspace.numel(),
                                        _stream(stream))
    else:
        name = "tdn_ablation_forward_atomics" if atomics_ablation else "tdn_cp_tp_forward"
        st = getattr(lib(), name)(ctypes.byref(p), _ptr(x), _ptr(edge_vec), _ptr(edge_index), _ptr(A), _ptr(B),
                                  _ptr(D), _ptr(W), _ptr(radial_w), _ptr(out), _ptr(z), _ptr(perm), _ptr(offsets),
                                  _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, name)
    return ForwardResult(out, z, perm, offsets, p,
                         dict(x=x, edge_vec=edge_vec, edge_index=edge_index, A=A, B=B, D=D, W=W, radial_w=radial_w))


ABL_FACTORS_GLOBAL, ABL_Y_TABLE, ABL_VALU = 1, 2, 3


def ablation_workspace_size(p: Problem, variant: int) -> int:
    """Workspace bytes of tdn_ablation_forward for this problem and variant."""
    nb = _SZ(0)
    _check(lib().tdn_ablation_workspace_size(ctypes.byref(p), int(variant), ctypes.byref(nb)),
           "tdn_ablation_workspace_size")
    return nb.value

NOALLOC_SCRATCH_BYTES = 32 << 20


def forward_noalloc(x, edge_vec, edge_index, A, B, D, W, radial_w, *, L: int, r_cut: float, out, perm, offsets,
                    z=None, edges_sorted=False, validate=False, stream=None) -> ForwardResult:
    """Runs tdn_cp_tp_forward_noalloc: the forward with the library's fixed
    scratch area instead of a workspace (for callers that cannot allocate).
    The outputs out, perm, offsets (and z, optional) must be passed
    preallocated; arguments otherwise as in forward()."""
    dev = x.device
    N, d, C = x.shape
    E = edge_vec.shape[0]
    R = A.shape[1]
    if edge_index.dtype != torch.int32 or not edge_index.is_contiguous():
        raise TypeError("edge_index must be contiguous int32 (no conversion happens on this path)")
    fd = TDN_BF16 if x.dtype == torch.bfloat16 else TDN_F32
    for t, n, dt, sh in [(x, "x", x.dtype, (N, d, C)), (edge_vec, "edge_vec", torch.float32, (E, 3)),
                         (edge_index, "edge_index", torch.int32, (2, E)), (A, "A", torch.float32, (d, R)),
                         (B, "B", torch.float32, (d, R)), (D, "D", torch.float32, (d, R)),
                         (W, "W", x.dtype, (C, C)), (radial_w, "radial_w", torch.float32, (radial_w.shape[0], R)),
                         (out, "out", torch.float32, (N, d, C)), (perm, "perm", torch.int32, (E,)),
                         (offsets, "offsets", torch.int32, (N + 1,))]:
        _need(t, n, dt, sh, dev)
    if z is not None:
        _need(z, "z", torch.float32, (N, d, C), dev)
    p = make_problem(L, C, R, N, E, r_cut, radial_w.shape[0], fd, edges_sorted, validate)
    st = lib().tdn_cp_tp_forward_noalloc(ctypes.byref(p), _ptr(x), _ptr(edge_vec), _ptr(edge_index), _ptr(A),
                                         _ptr(B), _ptr(D), _ptr(W), _ptr(radial_w), _ptr(out), _ptr(z), _ptr(perm),
                                         _ptr(offsets), _stream(stream))
    _check(st, "tdn_cp_tp_forward_noalloc")
    return ForwardResult(out, z, perm, offsets, p,
                         dict(x=x, edge_vec=edge_vec, edge_index=edge_index, A=A, B=B, D=D, W=W, radial_w=radial_w))


def forward3(x, edge_vec, edge_index, A, A2, B, D, W, radial_w, *, L: int, r_cut: float, edges_sorted=False,
             validate=False, workspace=None, out=None, z=None, perm=None, offsets=None,
             stream=None) -> ForwardResult:
    """Runs tdn_cp_tp3_forward, the three-input CP product whose third input
    is the destination node's features (A2 [d, R] its factor); float32
    features, 2 <= L <= 4.  Other arguments as in forward()."""
    dev = x.device
    N, d, C = x.shape
    E = edge_vec.shape[0]
    R = A.shape[1]
    if edge_index.dtype != torch.int32:
        edge_index = edge_index.to(torch.int32)
    edge_index = edge_index.contiguous()
    for t, n, dt, sh in [(x, "x", torch.float32, (N, d, C)), (edge_vec, "edge_vec", torch.float32, (E, 3)),
                         (edge_index, "edge_index", torch.int32, (2, E)), (A, "A", torch.float32, (d, R)),
                         (A2, "A2", torch.float32, (d, R)), (B, "B", torch.float32, (d, R)),
                         (D, "D", torch.float32, (d, R)), (W, "W", torch.float32, (C, C)),
                         (radial_w, "radial_w", torch.float32, (radial_w.shape[0], R))]:
        _need(t, n, dt, sh, dev)
    p = make_problem(L, C, R, N, E, r_cut, radial_w.shape[0], TDN_F32, edges_sorted, validate)
    fwd_bytes, _ = workspace_size(p)
    if workspace is None or workspace.numel() < fwd_bytes:
        workspace = torch.empty(max(fwd_bytes, 1), dtype=torch.uint8, device=dev)
    if out is None:
        out = torch.empty((N, d, C), dtype=torch.float32, device=dev)
    if perm is None:
        perm = torch.empty(max(E, 1), dtype=torch.int32, device=dev)[:E]
    if offsets is None:
        offsets = torch.empty(N + 1, dtype=torch.int32, device=dev)
    _need(out, "out", torch.float32, (N, d, C), dev)
    if z is not None:
        _need(z, "z", torch.float32, (N, d, C), dev)
    _need(perm, "perm", torch.int32, (E,), dev)
    _need(offsets, "offsets", torch.int32, (N + 1,), dev)
    st = lib().tdn_cp_tp3_forward(ctypes.byref(p), _ptr(x), _ptr(edge_vec), _ptr(edge_index), _ptr(A), _ptr(A2),
                                  _ptr(B), _ptr(D), _ptr(W), _ptr(radial_w), _ptr(out), _ptr(z), _ptr(perm),
                                  _ptr(offsets), _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "tdn_cp_tp3_forward")
    return ForwardResult(out, z, perm, offsets, p, dict(x=x, edge_vec=edge_vec, edge_index=edge_index, A=A, A2=A2,
                                                        B=B, D=D, W=W, radial_w=radial_w))


def ps_linear(x, W, *, workspace=None, out=None, stream=None):
    """Runs tdn_ps_linear: y = x W with one W [C, C] for every degree
    (path-weight-shared equivariant linear layer).  x [N, d, C] float32; W
    float32 or bfloat16."""
    dev = x.device
    N, d, C = x.shape
    L = int(round(d ** 0.5)) - 1
    if (L + 1) ** 2 != d:
        raise ValueError("x must be [N, (L+1)^2, C]")
    wd = TDN_BF16 if W.dtype == torch.bfloat16 else TDN_F32
    _need(x, "x", torch.float32, (N, d, C), dev)
    _need(W, "W", W.dtype, (C, C), dev)
    nb = _SZ()
    _check(lib().tdn_ps_linear_workspace_size(C, wd, ctypes.byref(nb)), "tdn_ps_linear_workspace_size")
    if workspace is None or workspace.numel() < nb.value:
        workspace = torch.empty(max(nb.value, 1), dtype=torch.uint8, device=dev)
    if out is None:
        out = torch.empty((N, d, C), dtype=torch.float32, device=dev)
    _need(out, "out", torch.float32, (N, d, C), dev)
    _check(lib().tdn_ps_linear(N, L, C, _ptr(x), _ptr(W), wd, _ptr(out), _ptr(workspace), workspace.numel(),
                               _stream(stream)), "tdn_ps_linear")
    return out


@dataclass
class CGTable:
    """The coefficient tensor in tdn_dense_tp_forward's row format (device
    tensors): row q = k d + i holds the entries (j | path << 16, value) of
    every nonzero C[k, i, j], in increasing j."""
    L: int
    n_path: int
    row: torch.Tensor
    col: torch.Tensor
    val: torch.Tensor


def cg_table(M, path, device) -> CGTable:
    """Marshals a dense coefficient tensor M [d, d, d] (index order k, i, j)
    and the path index of each entry ([d, d, d], -1 where M is zero) into the
    row format of tdn_dense_tp_forward."""
    import numpy as np

    M = np.asarray(M)
    path = np.asarray(path, np.int64)
    d = M.shape[0]
    L = int(round(d ** 0.5)) - 1
    if M.shape != (d, d, d) or path.shape != M.shape or (L + 1) ** 2 != d:
        raise ValueError("M and path must be [d, d, d] with d = (L + 1)^2")
    k, i, j = np.nonzero(M)                     # row-major: sorted by (k, i, j)
    p = path[k, i, j]
    if np.any(p < 0) or np.any(p >= 1 << 15):
        raise ValueError("every nonzero coefficient needs a path index in [0, 2^15)")
    q = k * d + i
    row = np.zeros(d * d + 1, np.int64)
    np.add.at(row, q + 1, 1)
    row = np.cumsum(row)
    col = (j | (p << 16)).astype(np.int32)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(device)  # noqa: E731
    return CGTable(L, int(path.max()) + 1 if path.size else 0, t(row.astype(np.int32)), t(col),
                   t(M[k, i, j].astype(np.float32)))


def dense_forward(x, edge_vec, edge_index, table: CGTable, path_w, W, *, r_cut: float, edges_sorted=False,
                  validate=False, workspace=None, out=None, z=None, perm=None, offsets=None,
                  stream=None) -> ForwardResult:
    """Runs tdn_dense_tp_forward, the exact CG tensor product over the same
    edges (float32 features).  path_w [n_radial, n_path] float32; the other
    arguments as in forward()."""
    dev = x.device
    N, d, C = x.shape
    E = edge_vec.shape[0]
    L = table.L
    P = path_w.shape[1]
    if edge_index.dtype != torch.int32:
        edge_index = edge_index.to(torch.int32)
    edge_index = edge_index.contiguous()
    for t, n, dt, sh in [(x, "x", torch.float32, (N, (L + 1) ** 2, C)), (edge_vec, "edge_vec", torch.float32, (E, 3)),
                         (edge_index, "edge_index", torch.int32, (2, E)), (W, "W", torch.float32, (C, C)),
                         (path_w, "path_w", torch.float32, (path_w.shape[0], P)),
                         (table.row, "table.row", torch.int32, (d * d + 1,)),
                         (table.col, "table.col", torch.int32, (table.col.shape[0],)),
                         (table.val, "table.val", torch.float32, (table.col.shape[0],))]:
        _need(t, n, dt, sh, dev)
    p = make_problem(L, C, P, N, E, r_cut, path_w.shape[0], TDN_F32, edges_sorted, validate)
    fwd_bytes, _ = workspace_size(p)
    if workspace is None or workspace.numel() < fwd_bytes:
        workspace = torch.empty(max(fwd_bytes, 1), dtype=torch.uint8, device=dev)
    if out is None:
        out = torch.empty((N, d, C), dtype=torch.float32, device=dev)
    if perm is None:
        perm = torch.empty(max(E, 1), dtype=torch.int32, device=dev)[:E]
    if offsets is None:
        offsets = torch.empty(N + 1, dtype=torch.int32, device=dev)
    _need(out, "out", torch.float32, (N, d, C), dev)
    if z is not None:
        _need(z, "z", torch.float32, (N, d, C), dev)
    _need(perm, "perm", torch.int32, (E,), dev)
    _need(offsets, "offsets", torch.int32, (N + 1,), dev)
    st = lib().tdn_dense_tp_forward(ctypes.byref(p), _ptr(x), _ptr(edge_vec), _ptr(edge_index), _ptr(table.row),
                                    _ptr(table.col), _ptr(table.val), int(table.col.shape[0]), _ptr(path_w), _ptr(W),
                                    _ptr(out), _ptr(z), _ptr(perm), _ptr(offsets), _ptr(workspace),
                                    workspace.numel(), _stream(stream))
    _check(st, "tdn_dense_tp_forward")
    return ForwardResult(out, z, perm, offsets, p, dict(x=x, edge_vec=edge_vec, edge_index=edge_index, W=W,
                                                        path_w=path_w))


def attention_workspace_size(p: Problem, n_heads: int, n_hidden: int) -> int:
    """Workspace bytes of tdn_attention_forward."""
    nb = _SZ(0)
    _check(lib().tdn_attention_workspace_size(ctypes.byref(p), int(n_heads), int(n_hidden), ctypes.byref(nb)),
           "tdn_attention_workspace_size")
    return nb.value


def attention_forward(x, edge_vec, edge_index, A, B, D, W, radial_w, att_w1, att_w2, *, L: int, r_cut: float,
                      edges_sorted=False, validate=False, workspace=None, out=None, z=None, alpha=None, perm=None,
                      offsets=None, stream=None):
    """Runs tdn_attention_forward (float32): att_w1 [2C + n_radial, F],
    att_w2 [F, H].  Returns (ForwardResult, alpha [E, H] by edge id)."""
    dev = x.device
    N, d, C = x.shape
    E = edge_vec.shape[0]
    R = A.shape[1]
    F, H = att_w2.shape
    if edge_index.dtype != torch.int32:
        edge_index = edge_index.to(torch.int32)
    edge_index = edge_index.contiguous()
    nr = radial_w.shape[0]
    for t, n, sh in [(x, "x", (N, d, C)), (edge_vec, "edge_vec", (E, 3)), (A, "A", (d, R)), (B, "B", (d, R)),
                     (D, "D", (d, R)), (W, "W", (C, C)), (radial_w, "radial_w", (nr, R)),
                     (att_w1, "att_w1", (2 * C + nr, F)), (att_w2, "att_w2", (F, H))]:
        _need(t, n, torch.float32, sh, dev)
    _need(edge_index, "edge_index", torch.int32, (2, E), dev)
    p = make_problem(L, C, R, N, E, r_cut, nr, TDN_F32, edges_sorted, validate)
    nbytes = attention_workspace_size(p, H, F)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    if out is None:
        out = torch.empty((N, d, C), dtype=torch.float32, device=dev)
    if alpha is None:
        alpha = torch.empty((E, H), dtype=torch.float32, device=dev)
    if perm is None:
        perm = torch.empty(max(E, 1), dtype=torch.int32, device=dev)[:E]
    if offsets is None:
        offsets = torch.empty(N + 1, dtype=torch.int32, device=dev)
    _need(out, "out", torch.float32, (N, d, C), dev)
    _need(alpha, "alpha", torch.float32, (E, H), dev)
    if z is not None:
        _need(z, "z", torch.float32, (N, d, C), dev)
    st = lib().tdn_attention_forward(ctypes.byref(p), int(H), int(F), _ptr(x), _ptr(edge_vec), _ptr(edge_index),
                                     _ptr(A), _ptr(B), _ptr(D), _ptr(W), _ptr(radial_w), _ptr(att_w1),
                                     _ptr(att_w2), _ptr(out), _ptr(alpha), _ptr(z), _ptr(perm), _ptr(offsets),
                                     _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "tdn_attention_forward")
    return ForwardResult(out, z, perm, offsets, p, dict(x=x, edge_vec=edge_vec, edge_index=edge_index, A=A, B=B,
                                                        D=D, W=W, radial_w=radial_w)), alpha


def dense_unshared_workspace_size(p: Problem) -> int:
    """Workspace bytes of tdn_dense_tp_forward_unshared for this problem."""
    nbytes = _SZ(0)
    _check(lib().tdn_dense_tp_unshared_workspace_size(ctypes.byref(p), ctypes.byref(nbytes)),
           "tdn_dense_tp_unshared_workspace_size")
    return nbytes.value


def dense_forward_unshared(x, edge_vec, edge_index, table: CGTable, path_w, W_paths, *, r_cut: float,
                           edges_sorted=False, validate=False, workspace=None, out=None, perm=None, offsets=None,
                           stream=None) -> ForwardResult:
    """Runs tdn_dense_tp_forward_unshared, the exact CG tensor product with one
    channel matrix per path (float32 features, C <= 128).  W_paths
    [n_path, C, C] float32 ([in][out] per path); the other arguments as in
    dense_forward()."""
    dev = x.device
    N, d, C = x.shape
    E = edge_vec.shape[0]
    L = table.L
    P = path_w.shape[1]
    if edge_index.dtype != torch.int32:
        edge_index = edge_index.to(torch.int32)
    edge_index = edge_index.contiguous()
    for t, n, dt, sh in [(x, "x", torch.float32, (N, (L + 1) ** 2, C)), (edge_vec, "edge_vec", torch.float32, (E, 3)),
                         (edge_index, "edge_index", torch.int32, (2, E)),
                         (W_paths, "W_paths", torch.float32, (P, C, C)),
                         (path_w, "path_w", torch.float32, (path_w.shape[0], P)),
                         (table.row, "table.row", torch.int32, (d * d + 1,)),
                         (table.col, "table.col", torch.int32, (table.col.shape[0],)),
                         (table.val, "table.val", torch.float32, (table.col.shape[0],))]:
        _need(t, n, dt, sh, dev)
    p = make_problem(L, C, P, N, E, r_cut, path_w.shape[0], TDN_F32, edges_sorted, validate)
    nbytes = dense_unshared_workspace_size(p)
    if workspace is None or workspace.numel() < nbytes:
        workspace = torch.empty(max(nbytes, 1), dtype=torch.uint8, device=dev)
    if out is None:
        out = torch.empty((N, d, C), dtype=torch.float32, device=dev)
    if perm is None:
        perm = torch.empty(max(E, 1), dtype=torch.int32, device=dev)[:E]
    if offsets is None:
        offsets = torch.empty(N + 1, dtype=torch.int32, device=dev)
    _need(out, "out", torch.float32, (N, d, C), dev)
    _need(perm, "perm", torch.int32, (E,), dev)
    _need(offsets, "offsets", torch.int32, (N + 1,), dev)
    st = lib().tdn_dense_tp_forward_unshared(ctypes.byref(p), _ptr(x), _ptr(edge_vec), _ptr(edge_index),
                                             _ptr(table.row), _ptr(table.col), _ptr(table.val),
                                             int(table.col.shape[0]), _ptr(path_w), _ptr(W_paths), _ptr(out),
                                             _ptr(perm), _ptr(offsets), _ptr(workspace), workspace.numel(),
                                             _stream(stream))
    _check(st, "tdn_dense_tp_forward_unshared")
    return ForwardResult(out, None, perm, offsets, p, dict(x=x, edge_vec=edge_vec, edge_index=edge_index,
                                                           W_paths=W_paths, path_w=path_w))


def backward(res: ForwardResult, grad_out, *, need_x=True, need_W=True, need_vec=True, need_radial=False,
             use_saved_z=True, workspace=None, stream=None):
    """Runs tdn_cp_tp_backward; returns (grad_x, grad_W, grad_edge_vec), each
    float32 or None, and grad_radial_w [n_radial, R] as a fourth value when
    need_radial is set."""
    i = res.inputs
    x = i["x"]
    dev = x.device
    N, d, C = x.shape
    E = i["edge_vec"].shape[0]
    _need(grad_out, "grad_out", torch.float32, (N, d, C), dev)
    p = res.problem
    _, bwd_bytes = workspace_size(p)
    if workspace is None or workspace.numel() < bwd_bytes:
        workspace = torch.empty(max(bwd_bytes, 1), dtype=torch.uint8, device=dev)
    gx = torch.empty((N, d, C), dtype=torch.float32, device=dev) if need_x else None
    gW = torch.empty((C, C), dtype=torch.float32, device=dev) if need_W else None
    gv = torch.empty((E, 3), dtype=torch.float32, device=dev) if need_vec else None
    gr = torch.empty(tuple(i["radial_w"].shape), dtype=torch.float32, device=dev) if need_radial else None
    z = res.z if use_saved_z else None
    st = lib().tdn_cp_tp_backward(ctypes.byref(p), _ptr(x), _ptr(i["edge_vec"]), _ptr(i["edge_index"]), _ptr(i["A"]),
                                  _ptr(i["B"]), _ptr(i["D"]), _ptr(i["W"]), _ptr(i["radial_w"]), _ptr(res.perm),
                                  _ptr(res.offsets), _ptr(z), _ptr(grad_out), _ptr(gx), _ptr(gW), _ptr(gv),
                                  _ptr(gr), _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "tdn_cp_tp_backward")
    return (gx, gW, gv, gr) if need_radial else (gx, gW, gv)


def sort_by_key(keys: torch.Tensor, n_keys: int, stream=None):
    """Stable sort of int32 keys in [0, n_keys): returns (perm, offsets)."""
    if keys.dtype != torch.int32 or not keys.is_contiguous():
        raise TypeError("keys must be contiguous int32")
    E = keys.numel()
    nb = _SZ()
    _check(lib().tdn_sort_workspace_size(int(n_keys), int(E), ctypes.byref(nb)), "tdn_sort_workspace_size")
    ws = torch.empty(max(nb.value, 1), dtype=torch.uint8, device=keys.device)
    perm = torch.empty(max(E, 1), dtype=torch.int32, device=keys.device)[:E]
    offsets = torch.empty(n_keys + 1, dtype=torch.int32, device=keys.device)
    _check(lib().tdn_sort_by_key(int(n_keys), int(E), _ptr(keys), _ptr(perm), _ptr(offsets), _ptr(ws), ws.numel(),
                                 _stream(stream)), "tdn_sort_by_key")
    return perm, offsets


@dataclass
class RadiusGraph:
    edge_index: torch.Tensor      # [2, E] int32, row 0 = src, row 1 = dst, sorted by (dst, src, image)
    edge_vec: torch.Tensor        # [E, 3] float32
    edge_image: torch.Tensor | None  # [E, 3] int32
    offsets: torch.Tensor         # [N+1] int32


def radius_graph(pos, graph_ptr, *, r_cut: float, cell=None, periodic=(False, False, False), max_neighbors=0,
                 capacity=None, want_image=False, workspace=None, stream=None) -> RadiusGraph:
    """Runs tdn_radius_graph.  pos [N,3] float32, graph_ptr [G+1] int32 (int64
    is converted), cell [G,3] float32 when an axis is periodic.  capacity:
    edge buffer size to try first (default: ask for the count, then build);
    a call with too small a capacity is repeated once with the exact count."""
    dev = pos.device
    N = pos.shape[0]
    if graph_ptr.dtype != torch.int32:
        graph_ptr = graph_ptr.to(torch.int32)
    graph_ptr = graph_ptr.contiguous()
    G = graph_ptr.numel() - 1
    _need(pos, "pos", torch.float32, (N, 3), dev)
    _need(graph_ptr, "graph_ptr", torch.int32, (G + 1,), dev)
    if cell is not None:
        _need(cell, "cell", torch.float32, (G, 3), dev)
    per = (ctypes.c_int32 * 3)(*[int(bool(p)) for p in periodic])
    g = GraphProblem(int(N), int(G), float(r_cut), int(max_neighbors), per)
    nb = _SZ()
    _check(lib().tdn_radius_graph_workspace_size(ctypes.byref(g), ctypes.byref(nb)), "tdn_radius_graph_workspace_size")
    if workspace is None or workspace.numel() < nb.value:
        workspace = torch.empty(max(nb.value, 1), dtype=torch.uint8, device=dev)
    offsets = torch.empty(N + 1, dtype=torch.int32, device=dev)
    n_edges = ctypes.c_int64()
    cap = 0 if capacity is None else int(capacity)
    for _ in range(2):
        ei = torch.empty(max(2 * cap, 1), dtype=torch.int32, device=dev)
        ev = torch.empty((max(cap, 1), 3), dtype=torch.float32, device=dev)
        im = torch.empty((max(cap, 1), 3), dtype=torch.int32, device=dev) if want_image else None
        st = lib().tdn_radius_graph(ctypes.byref(g), _ptr(pos), _ptr(graph_ptr), _ptr(cell), cap,
                                    _ptr(ei) if cap else None, _ptr(ev) if cap else None,
                                    _ptr(im) if cap and want_image else None, _ptr(offsets), ctypes.byref(n_edges),
                                    _ptr(workspace), workspace.numel(), _stream(stream))
        if st != TDN_ERR_EDGE_CAPACITY:
            break
        cap = n_edges.value
    _check(st, "tdn_radius_graph")
    E = n_edges.value
    return RadiusGraph(ei[:2 * E].view(2, E), ev[:E], im[:E] if want_image else None, offsets)


def spherical_harmonics(edge_vec: torch.Tensor, L: int, jacobian=False, stream=None):
    E = edge_vec.shape[0]
    _need(edge_vec, "edge_vec", torch.float32, (E, 3), edge_vec.device)
    d = (L + 1) ** 2
    Y = torch.empty((E, d), dtype=torch.float32, device=edge_vec.device)
    J = torch.empty((E, d, 3), dtype=torch.float32, device=edge_vec.device) if jacobian else None
    _check(lib().tdn_spherical_harmonics(int(L), int(E), _ptr(edge_vec), _ptr(Y), _ptr(J), _stream(stream)),
           "tdn_spherical_harmonics")
    return (Y, J) if jacobian else Y


def timer_enable(on: bool = True):
    _check(lib().tdn_timer_enable(int(bool(on))), "tdn_timer_enable")


def timer_read(kernel: str, reset=True) -> tuple[float, int]:
    ms, n = ctypes.c_double(), ctypes.c_int32()
    _check(lib().tdn_timer_read(kernel.encode(), ctypes.byref(ms), ctypes.byref(n), int(reset)), "tdn_timer_read")
    return ms.value, n.value
