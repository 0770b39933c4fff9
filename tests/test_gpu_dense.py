"""GPU parity of the exact CG tensor-product comparator (tdn_dense_tp_forward)
against the oracle's path-by-path layer (oracle/dense_layer.py), through the
C ABI.  Small problems are compared in full (Z and out); the headline-size
molecular workload at L = 4 and the L = 6 slab workload on sampled nodes.
The product without path-weight sharing (one channel matrix per path) is
checked against oracle dense_layer.forward_unshared the same way."""
import os

import numpy as np
import pytest
import torch

import paper_2507_01131_amd as tdn
import workloads
from oracle import cg_tensor, dense_layer, layer
from tests._gpu_helpers import TOL_F32, check_rows, rel_err, sample_nodes, workload

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


def _table(L):
    z = np.load(os.path.join(HERE, "golden", "cg", f"cg_L{L}.npz"))
    return tdn.cg_table(z["M"], z["path"], "cuda")


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _run(w, path_w, **kw):
    res = tdn.dense_forward(_t(w["x"]), _t(w["edge_vec"]), _t(w["edge_index"]), _table(w["L"]), _t(path_w),
                            _t(w["W"]), r_cut=w["r_cut"], edges_sorted=w["presorted"], **kw)
    torch.cuda.synchronize()
    return res


def _path_w(w, seed):
    P = len(cg_tensor.paths(w["L"]))
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((w["n_radial"], P)) / np.sqrt(w["n_radial"])).astype(np.float32)


SMALL = [
    # (L, C, N, E, sorted): every degree, channel counts with a ragged 32-wide tile
    # and two tiles per wave (C > 128), isolated nodes
    (0, 16, 30, 200, False), (1, 32, 40, 400, True), (2, 48, 50, 700, False), (3, 64, 60, 800, False),
    (4, 128, 70, 900, True), (4, 160, 40, 500, False), (5, 32, 40, 400, False), (6, 256, 30, 300, False),
    (6, 80, 25, 250, True),
]


@pytest.mark.parametrize("L,C,N,E,srt", SMALL, ids=lambda v: str(v))
def test_dense_small_full(L, C, N, E, srt):
    w = workloads.random_graph(300 + L + C, n_nodes=N, n_edges=E, L=L, C=C, R=1, sort=srt)
    pw = _path_w(w, L + C)
    z = torch.empty((N, (L + 1) ** 2, C), device="cuda")
    res = _run(w, pw, z=z)
    ref, refZ = dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], w["W"], pw, w["r_cut"], L,
                                    return_z=True)
    rp, ro = layer.stable_sort_by_key(w["edge_index"][1], N)
    np.testing.assert_array_equal(res.perm.cpu().numpy(), rp)
    np.testing.assert_array_equal(res.offsets.cpu().numpy(), ro)
    assert rel_err(z.cpu().numpy(), refZ) < TOL_F32
    assert rel_err(res.out.cpu().numpy(), ref) < TOL_F32


def test_dense_matches_the_cp_kernel_with_exact_per_path_factors():
    # two different GPU kernels, one result: the CP edge pass with factors
    # whose ranks each lie in one path (Thm. 2) and the exact product
    L = 2
    D, A, B, rank_path = dense_layer.exact_cp_factors(L)
    assert A.shape[1] <= 256
    w = workloads.random_graph(77, n_nodes=60, n_edges=900, L=L, C=64, R=1)
    pw = _path_w(w, 5)
    dense = _run(w, pw).out.cpu().numpy()
    f = lambda a: _t(a.astype(np.float32))  # noqa: E731
    cp = tdn.forward(_t(w["x"]), _t(w["edge_vec"]), _t(w["edge_index"]), f(A), f(B), f(D), _t(w["W"]),
                     f(pw[:, rank_path]), L=L, r_cut=w["r_cut"]).out.cpu().numpy()
    ref = dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], w["W"], pw, w["r_cut"], L)
    assert rel_err(dense, ref) < TOL_F32 and rel_err(cp, ref) < TOL_F32


def test_dense_no_edges_star_and_repeat_calls():
    L, C, N = 3, 64, 20
    w = workloads.random_graph(5, n_nodes=N, n_edges=0, L=L, C=C, R=1)
    out = _run(w, _path_w(w, 1)).out.cpu().numpy()
    assert np.all(out == 0)
    # a star: 700 edges into node 3 (many batches in one workgroup), none elsewhere
    w = workloads.random_graph(6, n_nodes=N, n_edges=700, L=L, C=C, R=1)
    w["edge_index"][1] = 3
    pw = _path_w(w, 2)
    a = _run(w, pw).out.cpu().numpy()
    b = _run(w, pw).out.cpu().numpy()
    np.testing.assert_array_equal(a, b)
    ref = dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], w["W"], pw, w["r_cut"], L)
    assert rel_err(a, ref) < TOL_F32
    assert np.all(a[np.arange(N) != 3] == 0)


def test_dense_zero_path_weights_give_zero():
    w = workloads.random_graph(8, n_nodes=30, n_edges=300, L=2, C=32, R=1)
    out = _run(w, np.zeros((w["n_radial"], 15), np.float32)).out.cpu().numpy()
    assert np.all(out == 0)


@pytest.mark.parametrize("name", ["molecules3200_L4_C128_R128", "slabs4960_L6_C128_R256"])
def test_dense_full_size_sampled(name):
    w = workload(name)
    pw = _path_w(w, 11)
    res = _run(w, pw)
    out = res.out.cpu().numpy()
    assert np.all(np.isfinite(out))
    nodes = sample_nodes(w, 16)
    perm, _ = layer.stable_sort_by_key(w["edge_index"][1], w["N"])
    keep = np.zeros(w["N"], bool)
    keep[nodes] = True
    sub = perm[keep[w["edge_index"][1][perm]]]
    ref = dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], w["W"], pw, w["r_cut"], w["L"], perm=sub)
    assert rel_err(out[nodes], ref[nodes]) < TOL_F32


@pytest.mark.parametrize("case,status", [("range", 5), ("order", 6), ("zero", 7)])
def test_dense_validation_errors(case, status):
    w = workloads.random_graph(12, n_nodes=10, n_edges=50, L=2, C=16, R=1, sort=True)
    if case == "range":
        w["edge_index"][0, 7] = 10
    elif case == "order":
        w["edge_index"][1, [3, 40]] = w["edge_index"][1, [40, 3]]
    else:
        w["edge_vec"][4] = 0
    with pytest.raises(tdn.TdnError) as ei:
        _run(w, _path_w(w, 1), validate=True)
    assert ei.value.status == status
    w2 = workloads.random_graph(12, n_nodes=10, n_edges=50, L=2, C=16, R=1, sort=True)
    _run(w2, _path_w(w2, 1), validate=True)          # good input passes


# ---- the product without path-weight sharing (tdn_dense_tp_forward_unshared)

def _w_paths(L, C, seed):
    P = len(cg_tensor.paths(L))
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((P, C, C)) / np.sqrt(C)).astype(np.float32)


def _run_un(w, path_w, W_paths, **kw):
    res = tdn.dense_forward_unshared(_t(w["x"]), _t(w["edge_vec"]), _t(w["edge_index"]), _table(w["L"]),
                                     _t(path_w), _t(W_paths), r_cut=w["r_cut"], edges_sorted=w["presorted"], **kw)
    torch.cuda.synchronize()
    return res


UNSHARED = [
    # (L, C, N, E, sorted): every degree (L = 4..6 in several row chunks),
    # ragged channel tiles, isolated nodes
    (0, 16, 30, 200, False), (1, 32, 40, 400, True), (2, 48, 50, 700, False), (3, 64, 60, 800, False),
    (4, 128, 70, 900, True), (4, 112, 40, 500, False), (5, 32, 40, 400, False), (6, 80, 25, 250, True),
]


@pytest.mark.parametrize("L,C,N,E,srt", UNSHARED, ids=lambda v: str(v))
def test_unshared_small_full(L, C, N, E, srt):
    w = workloads.random_graph(400 + L + C, n_nodes=N, n_edges=E, L=L, C=C, R=1, sort=srt)
    pw = _path_w(w, L + C + 1)
    Wp = _w_paths(L, C, L + C + 2)
    res = _run_un(w, pw, Wp)
    ref = dense_layer.forward_unshared(w["x"], w["edge_index"], w["edge_vec"], Wp, pw, w["r_cut"], L)
    rp, ro = layer.stable_sort_by_key(w["edge_index"][1], N)
    np.testing.assert_array_equal(res.perm.cpu().numpy(), rp)
    np.testing.assert_array_equal(res.offsets.cpu().numpy(), ro)
    out = res.out.cpu().numpy()
    assert rel_err(out, ref) < TOL_F32
    check_rows(out, ref, TOL_F32, "out")


@pytest.mark.parametrize("L", [2, 4])
def test_unshared_with_equal_path_matrices_is_the_shared_product(L):
    # one matrix W for every path: two GPU kernels (per-path sums then path
    # GEMMs, and the shared product's single node GEMM) give the same layer
    w = workloads.random_graph(90 + L, n_nodes=50, n_edges=800, L=L, C=64, R=1)
    pw = _path_w(w, 3)
    Wp = np.repeat(w["W"][None], len(cg_tensor.paths(L)), axis=0)
    un = _run_un(w, pw, Wp).out.cpu().numpy()
    sh = _run(w, pw).out.cpu().numpy()
    ref = dense_layer.forward(w["x"], w["edge_index"], w["edge_vec"], w["W"], pw, w["r_cut"], L)
    assert rel_err(un, ref) < TOL_F32 and rel_err(sh, ref) < TOL_F32
    check_rows(un, ref, TOL_F32, "out")


def test_unshared_single_path_matrix():
    # only path p carries a matrix: the output is that path's block alone,
    # nonzero in the rows of degree l3(p) only
    L, C = 3, 32
    w = workloads.random_graph(17, n_nodes=30, n_edges=400, L=L, C=C, R=1)
    pw = _path_w(w, 4)
    plist = cg_tensor.paths(L)
    p = plist.index((2, 1, 3))
    Wp = np.zeros((len(plist), C, C), np.float32)
    Wp[p] = _w_paths(L, C, 5)[p]
    out = _run_un(w, pw, Wp).out.cpu().numpy()
    ref = dense_layer.forward_unshared(w["x"], w["edge_index"], w["edge_vec"], Wp, pw, w["r_cut"], L)
    assert np.all(out[:, :9] == 0)
    assert rel_err(out, ref) < TOL_F32


def test_unshared_no_edges_star_and_repeat_calls():
    L, C, N = 4, 64, 20
    w = workloads.random_graph(7, n_nodes=N, n_edges=0, L=L, C=C, R=1)
    assert np.all(_run_un(w, _path_w(w, 1), _w_paths(L, C, 1)).out.cpu().numpy() == 0)
    w = workloads.random_graph(8, n_nodes=N, n_edges=600, L=L, C=C, R=1)
    w["edge_index"][1] = 5
    pw, Wp = _path_w(w, 2), _w_paths(L, C, 2)
    a = _run_un(w, pw, Wp).out.cpu().numpy()
    b = _run_un(w, pw, Wp).out.cpu().numpy()
    np.testing.assert_array_equal(a, b)
    ref = dense_layer.forward_unshared(w["x"], w["edge_index"], w["edge_vec"], Wp, pw, w["r_cut"], L)
    assert rel_err(a, ref) < TOL_F32
    assert np.all(a[np.arange(N) != 5] == 0)


def test_unshared_full_size_sampled():
    w = workload("molecules3200_L4_C128_R128")
    pw, Wp = _path_w(w, 12), _w_paths(w["L"], w["C"], 12)
    out = _run_un(w, pw, Wp).out.cpu().numpy()
    assert np.all(np.isfinite(out))
    nodes = sample_nodes(w, 16)
    perm, _ = layer.stable_sort_by_key(w["edge_index"][1], w["N"])
    keep = np.zeros(w["N"], bool)
    keep[nodes] = True
    sub = perm[keep[w["edge_index"][1][perm]]]
    ref = dense_layer.forward_unshared(w["x"], w["edge_index"], w["edge_vec"], Wp, pw, w["r_cut"], w["L"],
                                       perm=sub)
    assert rel_err(out[nodes], ref[nodes]) < TOL_F32
    check_rows(out[nodes], ref[nodes], TOL_F32, "out")
