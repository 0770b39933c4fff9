"""GPU radius graph against the brute-force oracle, through the C ABI.

Edge lists, images and offsets must match exactly and the float32 edge
vectors bit for bit (both sides round the same float32 operations in the same
order).  Small batches are compared in full; the five workloads' geometries
at full size on sampled destination atoms."""
import ctypes

import numpy as np
import pytest
import torch

import paper_2507_01131_amd as tdn
import workloads
from oracle import layer
from oracle import radius_graph as rg
from tests._gpu_helpers import TOL_F32, random_factors, rel_err

pytestmark = pytest.mark.gpu


def _gpu(inp, max_neighbors=0, capacity=None):
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    per = inp["periodic"]
    res = tdn.radius_graph(t(inp["pos"]), t(inp["graph_ptr"]), r_cut=inp["r_cut"],
                           cell=t(inp["cell"]) if any(per) else None, periodic=per, max_neighbors=max_neighbors,
                           capacity=capacity, want_image=True)
    torch.cuda.synchronize()
    return res


def _oracle(inp, max_neighbors=0, dst_nodes=None):
    return rg.radius_graph(inp["pos"], inp["graph_ptr"], inp["cell"] if any(inp["periodic"]) else None,
                           inp["periodic"], inp["r_cut"], max_neighbors=max_neighbors, dst_nodes=dst_nodes)


def _assert_same(res, ref, dsts=None):
    s, d, n, v = ref
    ei = res.edge_index.cpu().numpy()
    ev = res.edge_vec.cpu().numpy()
    im = res.edge_image.cpu().numpy()
    off = res.offsets.cpu().numpy()
    if dsts is None:
        np.testing.assert_array_equal(ei[0], s)
        np.testing.assert_array_equal(ei[1], d)
        np.testing.assert_array_equal(im, n)
        assert ev.tobytes() == v.tobytes()
        np.testing.assert_array_equal(off, np.searchsorted(d, np.arange(len(off)), side="left"))
        return
    for t in dsts:
        a, b = off[t], off[t + 1]
        sel = d == t
        np.testing.assert_array_equal(ei[0, a:b], s[sel])
        assert np.all(ei[1, a:b] == t)
        np.testing.assert_array_equal(im[a:b], n[sel])
        assert ev[a:b].tobytes() == v[sel].tobytes()


def _random_batch(seed, sizes, box, periodic, r_cut):
    rng = np.random.default_rng(seed)
    ptr = np.concatenate([[0], np.cumsum(sizes)])
    cell = np.array([[box * (1 + 0.1 * g), box, box * 0.9] for g in range(len(sizes))])
    pos = np.concatenate([rng.uniform(-0.5, 1.0, size=(n, 3)) * cell[g] for g, n in enumerate(sizes)])
    return workloads.wrap_inputs(pos, ptr, cell, periodic, r_cut)


SMALL = [
    dict(seed=1, sizes=[50, 0, 80, 1, 30], box=7.0, periodic=(True, True, True), r_cut=3.0),
    dict(seed=2, sizes=[200], box=10.0, periodic=(True, True, False), r_cut=4.0),
    dict(seed=3, sizes=[40, 60], box=6.0, periodic=(False, False, False), r_cut=2.5),
    dict(seed=4, sizes=[30, 25], box=4.0, periodic=(True, False, True), r_cut=3.5),     # boxes < 2 r_cut
    dict(seed=5, sizes=[300, 150], box=12.0, periodic=(True, True, True), r_cut=5.0),
    dict(seed=6, sizes=[5], box=3.0, periodic=(True, True, True), r_cut=2.6),          # one cell per axis
]


@pytest.mark.parametrize("cfg", SMALL, ids=lambda c: f"s{c['seed']}")
@pytest.mark.parametrize("cap", [0, 7])
def test_small_batches_exact(cfg, cap):
    inp = _random_batch(cfg["seed"], cfg["sizes"], cfg["box"], cfg["periodic"], cfg["r_cut"])
    res = _gpu(inp, max_neighbors=cap)
    ref = _oracle(inp, max_neighbors=cap)
    assert len(ref[0]) > 0
    _assert_same(res, ref)


@pytest.mark.parametrize("name", list(workloads.WORKLOADS))
def test_workload_geometries_full_size_sampled(name):
    inp = workloads.graph_inputs(name)
    res = _gpu(inp)
    N = inp["pos"].shape[0]
    off = res.offsets.cpu().numpy()
    ei = res.edge_index.cpu().numpy()
    assert off[0] == 0 and off[-1] == ei.shape[1] and np.all(np.diff(off) >= 0)
    assert np.all(np.diff(ei[1]) >= 0)
    rng = np.random.default_rng(1)
    dsts = np.sort(rng.choice(N, min(N, 96), replace=False))
    _assert_same(res, _oracle(inp, dst_nodes=dsts), dsts)
    # the fixture graph (float64 decisions) differs only at pairs on the cutoff
    E_fix = workloads.make_workload(name)["E"]
    assert abs(ei.shape[1] - E_fix) <= max(2, E_fix // 100000)


@pytest.mark.parametrize("r_cut,cap", [(5.0, 500), (12.0, 20)])
def test_oc20_and_oc22_cutoffs_and_caps_on_the_bulk_geometry(r_cut, cap):
    inp = dict(workloads.graph_inputs("bulk4096_L4_C256_R128_bf16"), r_cut=r_cut)
    res = _gpu(inp, max_neighbors=cap)
    counts = np.diff(res.offsets.cpu().numpy())
    N = inp["pos"].shape[0]
    rng = np.random.default_rng(2)
    dsts = np.sort(rng.choice(N, 48, replace=False))
    ref = _oracle(inp, max_neighbors=cap, dst_nodes=dsts)
    _assert_same(res, ref, dsts)
    if cap == 20:
        assert np.all(counts == 20)


def test_capacity_protocol_and_errors():
    inp = _random_batch(7, [100], 8.0, (True, True, True), 3.0)
    ref = _oracle(inp)
    E = len(ref[0])
    _assert_same(_gpu(inp, capacity=E // 3), ref)          # too small: retried with the count
    _assert_same(_gpu(inp, capacity=E + 100), ref)         # larger buffers: first E used
    pos = torch.from_numpy(inp["pos"]).cuda()
    ptr = torch.from_numpy(inp["graph_ptr"]).cuda()
    cell = torch.from_numpy(inp["cell"]).cuda()
    g = tdn.GraphProblem(100, 1, 3.0, 0, (ctypes.c_int32 * 3)(1, 1, 1))
    nb = ctypes.c_size_t()
    assert tdn.lib().tdn_radius_graph_workspace_size(ctypes.byref(g), ctypes.byref(nb)) == 0
    ws = torch.empty(nb.value, dtype=torch.uint8, device="cuda")
    ei = torch.empty(2 * E, dtype=torch.int32, device="cuda")
    ev = torch.empty((E, 3), dtype=torch.float32, device="cuda")
    n = ctypes.c_int64()

    def call(p, c, cap):
        return tdn.lib().tdn_radius_graph(ctypes.byref(g), ctypes.c_void_p(p.data_ptr()),
                                          ctypes.c_void_p(ptr.data_ptr()), ctypes.c_void_p(c.data_ptr()), cap,
                                          ctypes.c_void_p(ei.data_ptr()), ctypes.c_void_p(ev.data_ptr()), None,
                                          None, ctypes.byref(n), ctypes.c_void_p(ws.data_ptr()), ws.numel(), None)
    assert call(pos, cell, E - 1) == 11 and n.value == E
    assert call(pos, cell, E) == 0 and n.value == E
    bad = pos.clone()
    bad[17, 1] = cell[0, 1]                                  # coordinate == L: outside [0, L)
    assert call(bad, cell, E) == 10
    bad[17, 1] = float("nan")
    assert call(bad, cell, E) == 10
    assert call(pos, torch.full_like(cell, 2.0), E) == 10    # box shorter than r_cut
    torch.cuda.synchronize()


def test_inconsistent_graph_ptr_and_neighbour_limit():
    with pytest.raises(tdn.TdnError) as ei:
        tdn.radius_graph(torch.zeros((10, 3), device="cuda") + torch.arange(10, device="cuda")[:, None],
                         torch.tensor([0, 4, 9], dtype=torch.int32, device="cuda"), r_cut=2.0)
    assert ei.value.status == 10
    rng = np.random.default_rng(4)
    dense = torch.from_numpy(rng.uniform(0, 1.0, size=(2100, 3)).astype(np.float32)).cuda()
    with pytest.raises(tdn.TdnError) as ei:
        tdn.radius_graph(dense, torch.tensor([0, 2100], dtype=torch.int32, device="cuda"), r_cut=2.0)
    assert ei.value.status == 12
    res = tdn.radius_graph(dense[:2000], torch.tensor([0, 2000], dtype=torch.int32, device="cuda"), r_cut=2.0,
                           max_neighbors=16)
    torch.cuda.synchronize()
    assert res.edge_index.shape[1] == 2000 * 16
    res = tdn.radius_graph(torch.zeros((0, 3), device="cuda"), torch.zeros(1, dtype=torch.int32, device="cuda"),
                           r_cut=2.0)
    assert res.edge_index.shape == (2, 0)


def test_built_graph_feeds_the_layer():
    inp = _random_batch(8, [60, 40], 8.0, (True, True, False), 3.5)
    res = _gpu(inp)
    s, d, n, v = _oracle(inp)
    N, E, L, C, R = 100, len(s), 3, 32, 32
    A, B, D = random_factors(L, R, 8)
    rng = np.random.default_rng(8)
    x = rng.standard_normal((N, 16, C)).astype(np.float32)
    W = (rng.standard_normal((C, C)) / np.sqrt(C)).astype(np.float32)
    rw = (rng.standard_normal((8, R)) / np.sqrt(8)).astype(np.float32)
    c = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    out = tdn.forward(c(x), res.edge_vec, res.edge_index, c(A), c(B), c(D), c(W), c(rw), L=L, r_cut=3.5,
                      edges_sorted=True).out
    torch.cuda.synchronize()
    ref = layer.forward(x, np.stack([s, d]).astype(np.int32), v, A, B, D, W, rw, 3.5, L)
    assert rel_err(out.cpu(), ref) < TOL_F32


def test_grid_limits_and_cell_boundaries():
    rng = np.random.default_rng(21)
    # (a) clusters spread over 1e5 A: the 1024-cells-per-axis and 2 n + 1
    # cells-per-system bounds widen the cells far beyond the cutoff
    centres = rng.uniform(0, 1e5, size=(20, 3))
    pos = np.concatenate([c + rng.uniform(0, 6.0, size=(25, 3)) for c in centres])
    inp = workloads.wrap_inputs(pos, [0, len(pos)], np.zeros((1, 3)), (False, False, False), 3.0)
    _assert_same(_gpu(inp), _oracle(inp))
    # (b) a lattice whose spacing is the smallest cell width the grid allows
    # (1.001 r_cut), so atoms sit on cell boundaries, plus the same lattice
    # shifted by half a spacing along x (two neighbours at 1.001 per atom);
    # periodic and open axes
    r_cut = 2.0
    a = np.float32(r_cut * 1.001)
    n = 9
    g = np.stack(np.meshgrid(*[np.arange(n)] * 3, indexing="ij"), -1).reshape(-1, 3) * float(a)
    g2 = np.concatenate([g, g + np.array([0.5 * float(a), 0.0, 0.0])])
    jitter = rng.choice([0.0, 1e-6, -1e-6], size=g2.shape)
    L = float(np.float32(n * a))
    for per in [(True, True, True), (True, False, False)]:
        inp = workloads.wrap_inputs(g2 + jitter, [0, len(g2)], np.array([[L, L, L]]), per, r_cut)
        ref = _oracle(inp)
        assert len(ref[0]) > 0
        _assert_same(_gpu(inp), ref)
    # (c) spacing just under the cutoff: every lattice neighbour is an edge
    inp = workloads.wrap_inputs(g * (1.9 / float(a)), [0, len(g)], np.array([[9 * 1.9] * 3]), (True,) * 3, r_cut)
    res = _gpu(inp)
    assert res.edge_index.shape[1] == 6 * len(g)
    _assert_same(res, _oracle(inp))


def test_large_periodic_system_sampled():
    rng = np.random.default_rng(22)
    N, box = 20000, 58.0
    inp = workloads.wrap_inputs(rng.uniform(0, box, size=(N, 3)), [0, N], np.array([[box, box, box]]),
                                (True, True, True), 4.0)
    res = _gpu(inp, max_neighbors=24)
    dsts = np.sort(rng.choice(N, 64, replace=False))
    _assert_same(res, _oracle(inp, max_neighbors=24, dst_nodes=dsts), dsts)
