"""GPU parity of the three-input CP product (tdn_cp_tp3_forward: source
features, edge harmonics, destination features; App. A with N = 3) against
the oracle's per-edge layer.forward3, through the C ABI."""
import numpy as np
import pytest
import torch

import paper_2507_01131_amd as tdn
import workloads
from oracle import layer
from tests._gpu_helpers import TOL_F32, load_factors, rel_err, random_factors, sample_nodes, workload

pytestmark = pytest.mark.gpu


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _a2(L, R, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal(((L + 1) ** 2, R)) / (L + 1)).astype(np.float32)


def _run(w, A, A2, B, D, **kw):
    res = tdn.forward3(_t(w["x"]), _t(w["edge_vec"]), _t(w["edge_index"]), _t(A), _t(A2), _t(B), _t(D), _t(w["W"]),
                       _t(w["radial_w"]), L=w["L"], r_cut=w["r_cut"], edges_sorted=w["presorted"], **kw)
    torch.cuda.synchronize()
    return res


SMALL = [(2, 32, 32, 40, 600, True), (2, 48, 40, 50, 700, False), (3, 64, 64, 60, 900, False),
         (4, 128, 128, 70, 1000, True), (4, 32, 100, 30, 400, False)]


@pytest.mark.parametrize("L,C,R,N,E,srt", SMALL, ids=lambda v: str(v))
def test_three_input_small_full(L, C, R, N, E, srt):
    w = workloads.random_graph(500 + L + C, n_nodes=N, n_edges=E, L=L, C=C, R=R, sort=srt)
    A, B, D = random_factors(L, R, 7 + L)
    A2 = _a2(L, R, 9 + L)
    z = torch.empty((N, (L + 1) ** 2, C), device="cuda")
    res = _run(w, A, A2, B, D, z=z)
    ref = layer.forward3(w["x"], w["edge_index"], w["edge_vec"], A, A2, B, D, w["W"], w["radial_w"], w["r_cut"], L)
    rp, ro = layer.stable_sort_by_key(w["edge_index"][1], N)
    np.testing.assert_array_equal(res.perm.cpu().numpy(), rp)
    np.testing.assert_array_equal(res.offsets.cpu().numpy(), ro)
    assert rel_err(res.out.cpu().numpy(), ref) < TOL_F32
    assert np.allclose(z.cpu().numpy() @ w["W"], res.out.cpu().numpy(), rtol=1e-4, atol=1e-4 * np.abs(ref).max())


def test_three_input_hub_spans_edge_ranges():
    # 90 % of 6000 edges into node 2: that segment crosses many edge ranges,
    # so its partial sums are multiplied by A2^T x[2] before they are added
    L, C, R, N, E = 3, 64, 64, 50, 6000
    w = workloads.random_graph(21, n_nodes=N, n_edges=E, L=L, C=C, R=R)
    hub = np.random.default_rng(3).random(E) < 0.9
    w["edge_index"][1][hub] = 2
    A, B, D = random_factors(L, R, 11)
    A2 = _a2(L, R, 12)
    got = _run(w, A, A2, B, D).out.cpu().numpy()
    ref = layer.forward3(w["x"], w["edge_index"], w["edge_vec"], A, A2, B, D, w["W"], w["radial_w"], w["r_cut"], L)
    assert rel_err(got, ref) < TOL_F32
    assert rel_err(got[2], ref[2]) < TOL_F32


def test_three_input_with_constant_third_factor_matches_the_two_input_kernel():
    L, C, R = 4, 128, 128
    w = workloads.random_graph(31, n_nodes=80, n_edges=1500, L=L, C=C, R=R)
    w["x"][:, 0, :] = 1.0
    A, B, D = random_factors(L, R, 13)
    A2 = np.zeros_like(A)
    A2[0, :] = 1.0
    got = _run(w, A, A2, B, D).out.cpu().numpy()
    two = tdn.forward(_t(w["x"]), _t(w["edge_vec"]), _t(w["edge_index"]), _t(A), _t(B), _t(D), _t(w["W"]),
                      _t(w["radial_w"]), L=L, r_cut=w["r_cut"]).out.cpu().numpy()
    ref = layer.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], w["r_cut"], L)
    assert rel_err(got, ref) < TOL_F32 and rel_err(two, ref) < TOL_F32


def test_three_input_no_edges_and_repeat_calls():
    L, C, R = 2, 32, 32
    w = workloads.random_graph(41, n_nodes=20, n_edges=0, L=L, C=C, R=R)
    A, B, D = random_factors(L, R, 1)
    A2 = _a2(L, R, 2)
    assert np.all(_run(w, A, A2, B, D).out.cpu().numpy() == 0)
    w = workloads.random_graph(42, n_nodes=60, n_edges=2000, L=L, C=C, R=R)
    a = _run(w, A, A2, B, D).out.cpu().numpy()
    b = _run(w, A, A2, B, D).out.cpu().numpy()
    np.testing.assert_array_equal(a, b)


def test_three_input_headline_size_sampled():
    w = workload("molecules3200_L4_C128_R128")
    A, B, D = load_factors(w["L"], w["R"])
    A2 = _a2(w["L"], w["R"], 5)
    out = _run(w, A, A2, B, D).out.cpu().numpy()
    nodes = sample_nodes(w, 16)
    perm, _ = layer.stable_sort_by_key(w["edge_index"][1], w["N"])
    keep = np.zeros(w["N"], bool)
    keep[nodes] = True
    sub = perm[keep[w["edge_index"][1][perm]]]
    ref = layer.forward3(w["x"], w["edge_index"], w["edge_vec"], A, A2, B, D, w["W"], w["radial_w"], w["r_cut"],
                         w["L"], perm=sub)
    assert rel_err(out[nodes], ref[nodes]) < TOL_F32


@pytest.mark.parametrize("case,status", [("range", 5), ("order", 6), ("zero", 7)])
def test_three_input_validation_errors(case, status):
    L, R = 2, 32
    w = workloads.random_graph(13, n_nodes=10, n_edges=50, L=L, C=16, R=R, sort=True)
    A, B, D = random_factors(L, R, 3)
    A2 = _a2(L, R, 4)
    if case == "range":
        w["edge_index"][0, 7] = 10
    elif case == "order":
        w["edge_index"][1, [3, 40]] = w["edge_index"][1, [40, 3]]
    else:
        w["edge_vec"][4] = 0
    with pytest.raises(tdn.TdnError) as ei:
        _run(w, A, A2, B, D, validate=True)
    assert ei.value.status == status
