"""The forward and backward calls captured in a HIP graph (through
torch.cuda.CUDAGraph on the capture stream the library is handed).

Each replay is checked against the eager result bit for bit (the layer is
deterministic), with eager work and synchronisations between the replays,
and after the captured inputs are overwritten in place."""
import numpy as np
import pytest
import torch

import paper_2507_01131_amd as tdn
import workloads
from tests._gpu_helpers import random_factors

pytestmark = pytest.mark.gpu


def _inputs(seed, N, E, L, C, R, sort):
    w = workloads.random_graph(seed, n_nodes=N, n_edges=E, L=L, C=C, R=R, sort=sort)
    A, B, D = random_factors(L, R, seed)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).cuda()  # noqa: E731
    return w, dict(x=t(w["x"]), edge_vec=t(w["edge_vec"]), edge_index=t(w["edge_index"]), A=t(A), B=t(B), D=t(D),
                   W=t(w["W"]), radial_w=t(w["radial_w"]))


@pytest.mark.parametrize("N,E,L,C,R,sort", [(40, 900, 2, 32, 32, True), (120, 3000, 4, 128, 128, False)])
def test_forward_and_backward_replays_match_eager(N, E, L, C, R, sort):
    w, inp = _inputs(11 + L, N, E, L, C, R, sort)
    d = (L + 1) ** 2
    args = [inp[k] for k in ("x", "edge_vec", "edge_index", "A", "B", "D", "W", "radial_w")]
    p = tdn.make_problem(L, C, R, N, E, w["r_cut"], w["n_radial"], tdn.TDN_F32, sort)
    fb, bb = tdn.workspace_size(p)
    ws = torch.empty(fb, dtype=torch.uint8, device="cuda")
    wsb = torch.empty(bb, dtype=torch.uint8, device="cuda")
    out = torch.empty((N, d, C), device="cuda")
    z = torch.empty((N, d, C), device="cuda")
    perm = torch.empty(E, dtype=torch.int32, device="cuda")
    off = torch.empty(N + 1, dtype=torch.int32, device="cuda")
    G = torch.from_numpy(w["grad_out"]).cuda()

    def step():
        res = tdn.forward(*args, L=L, r_cut=w["r_cut"], edges_sorted=sort, workspace=ws, out=out, z=z, perm=perm,
                          offsets=off)
        return res, tdn.backward(res, G, workspace=wsb, need_radial=True)

    res, grads = step()                              # eager, also warms up the library
    torch.cuda.synchronize()
    ref = [out.clone(), z.clone(), perm.clone(), off.clone()] + [g.clone() for g in grads]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()                                       # warm-up on the side stream before capture
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _, gg = step()
    for k in range(4):
        out.zero_()
        z.zero_()
        for t in gg:
            t.zero_()
        g.replay()
        torch.cuda.synchronize()
        now = [out, z, perm, off] + list(gg)
        for a, b in zip(now, ref):
            assert torch.equal(a, b), k
        # eager work of other shapes between replays
        other = torch.randn(1000, 1000, device="cuda")
        (other @ other).sum().item()
    # new input values in the captured buffers: the replay computes with them
    inp["x"].copy_(torch.randn_like(inp["x"]))
    g.replay()
    torch.cuda.synchronize()
    got = out.clone()
    eager = tdn.forward(*args, L=L, r_cut=w["r_cut"], edges_sorted=sort).out
    torch.cuda.synchronize()
    assert torch.equal(got, eager) and not torch.equal(got, ref[0])


def _replays_match(call, outs, k=3):
    """Captures call() once, replays it k times with the outputs cleared and
    eager work in between, and compares every replay bit for bit with the
    eager result."""
    call()
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        call()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    for i in range(k):
        for o in outs:
            o.zero_()
        g.replay()
        torch.cuda.synchronize()
        for a, b in zip(outs, ref):
            assert torch.equal(a, b), i
        other = torch.randn(700, 700, device="cuda")
        (other @ other).sum().item()


def test_exact_comparator_and_three_input_replays_match_eager():
    import os

    L, C, R, N, E = 3, 64, 64, 60, 1500
    w, inp = _inputs(17, N, E, L, C, R, False)
    d = (L + 1) ** 2
    out = torch.empty((N, d, C), device="cuda")
    perm = torch.empty(E, dtype=torch.int32, device="cuda")
    off = torch.empty(N + 1, dtype=torch.int32, device="cuda")
    A2 = torch.from_numpy(random_factors(L, R, 99)[0]).cuda()
    p = tdn.make_problem(L, C, R, N, E, w["r_cut"], w["n_radial"], tdn.TDN_F32, False)
    ws = torch.empty(tdn.workspace_size(p)[0], dtype=torch.uint8, device="cuda")
    args = [inp[k] for k in ("x", "edge_vec", "edge_index", "A")] + [A2] + [inp[k] for k in ("B", "D", "W", "radial_w")]
    _replays_match(lambda: tdn.forward3(*args, L=L, r_cut=w["r_cut"], workspace=ws, out=out, perm=perm,
                                        offsets=off), [out, perm, off])
    z = np.load(os.path.join(os.path.dirname(__file__), "golden", "cg", f"cg_L{L}.npz"))
    tab = tdn.cg_table(z["M"], z["path"], "cuda")
    pw = torch.from_numpy(np.random.default_rng(3).standard_normal((w["n_radial"], tab.n_path)).astype(np.float32))
    pw = pw.cuda()
    pd = tdn.make_problem(L, C, tab.n_path, N, E, w["r_cut"], w["n_radial"], tdn.TDN_F32, False)
    wsd = torch.empty(tdn.workspace_size(pd)[0], dtype=torch.uint8, device="cuda")
    _replays_match(lambda: tdn.dense_forward(inp["x"], inp["edge_vec"], inp["edge_index"], tab, pw, inp["W"],
                                             r_cut=w["r_cut"], workspace=wsd, out=out, perm=perm, offsets=off),
                   [out, perm, off])
