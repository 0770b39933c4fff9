"""GPU parity of the attention block (tdn_attention_forward) against the
oracle (oracle/attention.py), through the C ABI: output, the saved weighted
sum and the attention weights on small problems in full (every degree it
supports, 1 to 4 heads, sorted and unsorted edges), the headline molecular
workload on sampled nodes, the mean-aggregation special case against the
plain CP forward, degenerate graphs, repeat calls and argument errors."""
import numpy as np
import pytest
import torch

import paper_2507_01131_amd as tdn
import workloads
from oracle import attention, layer
from tests._gpu_helpers import TOL_F32, check_rows, load_factors, random_factors, rel_err, sample_nodes, workload

pytestmark = pytest.mark.gpu


def _t(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def _att_weights(C, n_radial, F, H, seed, scale=2.0):
    rng = np.random.default_rng(seed)
    W1 = (scale * rng.standard_normal((2 * C + n_radial, F)) / np.sqrt(2 * C + n_radial)).astype(np.float32)
    w2 = (scale * rng.standard_normal((F, H)) / np.sqrt(F)).astype(np.float32)
    return W1, w2


def _run(w, A, B, D, W1, w2, **kw):
    res, alpha = tdn.attention_forward(_t(w["x"]), _t(w["edge_vec"]), _t(w["edge_index"]), _t(A), _t(B), _t(D),
                                       _t(w["W"]), _t(w["radial_w"]), _t(W1), _t(w2), L=w["L"], r_cut=w["r_cut"],
                                       edges_sorted=w["presorted"], **kw)
    torch.cuda.synchronize()
    return res, alpha


CASES = [
    # (seed, L, C, R, H, F, N, E, sorted)
    (1, 1, 32, 32, 1, 8, 30, 300, False), (2, 2, 64, 32, 2, 16, 40, 600, True), (3, 3, 64, 64, 2, 32, 50, 800, False),
    (4, 4, 128, 128, 4, 32, 60, 1200, False), (5, 4, 128, 100, 1, 64, 40, 700, True), (6, 2, 128, 48, 4, 7, 35, 500,
                                                                                         False),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: f"L{c[1]}C{c[2]}R{c[3]}H{c[4]}F{c[5]}")
def test_attention_small_full(case):
    seed, L, C, R, H, F, N, E, srt = case
    w = workloads.random_graph(600 + seed, n_nodes=N, n_edges=E, L=L, C=C, R=R, sort=srt)
    A, B, D = random_factors(L, R, seed)
    W1, w2 = _att_weights(C, w["n_radial"], F, H, seed)
    z = torch.empty((N, (L + 1) ** 2, C), device="cuda")
    res, alpha = _run(w, A, B, D, W1, w2, z=z)
    ref, ralpha, rz = attention.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], W1,
                                        w2, w["r_cut"], L, return_z=True)
    rp, ro = layer.stable_sort_by_key(w["edge_index"][1], N)
    np.testing.assert_array_equal(res.perm.cpu().numpy(), rp)
    np.testing.assert_array_equal(res.offsets.cpu().numpy(), ro)
    a = alpha.cpu().numpy()
    assert np.max(np.abs(a - ralpha) / ralpha) < 1e-5
    out = res.out.cpu().numpy()
    assert rel_err(out, ref) < TOL_F32
    check_rows(out, ref, TOL_F32, "out")
    check_rows(z.cpu().numpy(), rz, TOL_F32, "z")


def test_constant_logits_give_the_cp_forward_over_the_in_degree():
    # two GPU paths: zero attention weights give the mean of the messages,
    # the plain forward's output divided by each node's in-degree
    w = workloads.random_graph(77, n_nodes=50, n_edges=900, L=3, C=64, R=64)
    A, B, D = random_factors(3, 64, 77)
    W1 = np.zeros((2 * 64 + w["n_radial"], 8), np.float32)
    w2 = np.zeros((8, 2), np.float32)
    res, alpha = _run(w, A, B, D, W1, w2)
    plain = tdn.forward(_t(w["x"]), _t(w["edge_vec"]), _t(w["edge_index"]), _t(A), _t(B), _t(D), _t(w["W"]),
                        _t(w["radial_w"]), L=3, r_cut=w["r_cut"]).out.cpu().numpy().astype(np.float64)
    deg = np.bincount(w["edge_index"][1], minlength=50).astype(np.float64)
    np.testing.assert_allclose(alpha.cpu().numpy(), (1.0 / deg[w["edge_index"][1]])[:, None].repeat(2, 1),
                               rtol=1e-6)
    assert rel_err(res.out.cpu().numpy(), plain / np.maximum(deg, 1)[:, None, None]) < TOL_F32


def test_attention_headline_size_sampled():
    w = workload("molecules3200_L4_C128_R128")
    A, B, D = load_factors(w["L"], w["R"])
    W1, w2 = _att_weights(w["C"], w["n_radial"], 32, 4, 9)
    res, alpha = _run(w, A, B, D, W1, w2)
    out = res.out.cpu().numpy()
    assert np.all(np.isfinite(out))
    nodes = sample_nodes(w, 16)
    perm, _ = layer.stable_sort_by_key(w["edge_index"][1], w["N"])
    keep = np.zeros(w["N"], bool)
    keep[nodes] = True
    sub = perm[keep[w["edge_index"][1][perm]]]
    ref, ralpha = attention.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], W1, w2,
                                    w["r_cut"], w["L"], perm=sub)
    a = alpha.cpu().numpy()
    assert np.max(np.abs(a - ralpha) / ralpha) < 1e-5      # every edge's weights
    assert rel_err(out[nodes], ref[nodes]) < TOL_F32
    check_rows(out[nodes], ref[nodes], TOL_F32, "out")


def test_attention_no_edges_star_and_repeat_calls():
    L, C, N = 2, 64, 20
    A, B, D = random_factors(L, 32, 5)
    w = workloads.random_graph(5, n_nodes=N, n_edges=0, L=L, C=C, R=32)
    W1, w2 = _att_weights(C, w["n_radial"], 8, 2, 5)
    res, _ = _run(w, A, B, D, W1, w2)
    assert np.all(res.out.cpu().numpy() == 0)
    # a star: 700 edges into node 3 (the softmax runs over eleven lane passes)
    w = workloads.random_graph(6, n_nodes=N, n_edges=700, L=L, C=C, R=32)
    w["edge_index"][1] = 3
    r1, a1 = _run(w, A, B, D, W1, w2)
    r2, a2 = _run(w, A, B, D, W1, w2)
    np.testing.assert_array_equal(r1.out.cpu().numpy(), r2.out.cpu().numpy())
    np.testing.assert_array_equal(a1.cpu().numpy(), a2.cpu().numpy())
    ref, ralpha = attention.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], W1, w2,
                                    w["r_cut"], L)
    assert rel_err(r1.out.cpu().numpy(), ref) < TOL_F32
    assert np.max(np.abs(a1.cpu().numpy() - ralpha) / ralpha) < 1e-5
    assert np.all(r1.out.cpu().numpy()[np.arange(N) != 3] == 0)


@pytest.mark.parametrize("bad,status", [("heads", 2), ("degree", 2), ("hidden", 2)])
def test_attention_rejects_unsupported_problems(bad, status):
    L, C, H, F = 2, 64, 2, 8
    if bad == "heads":
        H = 4            # C = 64 is not a multiple of 32 * 4
    if bad == "degree":
        L = 5
    if bad == "hidden":
        F = 65
    w = workloads.random_graph(8, n_nodes=10, n_edges=40, L=L, C=C, R=32)
    A, B, D = random_factors(L, 32, 8)
    W1, w2 = _att_weights(C, w["n_radial"], F, H, 8)
    with pytest.raises(tdn.TdnError) as ei:
        _run(w, A, B, D, W1, w2)
    assert ei.value.status == status
