"""tdn_cp_tp_forward_noalloc, the forward for callers that cannot allocate,
against tdn_cp_tp_forward (the same launches on a caller's workspace) through
the C ABI: two calls in a row on one device, the second on a smaller
problem, must give the same bits as the workspace forward and match the
oracle within the float32 tolerance.  Outputs start filled with NaN so that
a region the call failed to write shows up."""
import numpy as np
import pytest
import torch

import paper_2507_01131_amd as tdn
import workloads
from oracle import layer
from tests._gpu_helpers import TOL_F32, check_rows, load_factors, random_factors, rel_err

pytestmark = pytest.mark.gpu


def _run_both(w, A, B, D):
    dev = "cuda"
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    args = (t(w["x"]), t(w["edge_vec"]), t(w["edge_index"]), t(A), t(B), t(D), t(w["W"]), t(w["radial_w"]))
    ref = tdn.forward(*args, L=w["L"], r_cut=w["r_cut"], edges_sorted=w["presorted"])
    N, d, C, E = w["N"], w["d"], w["C"], w["E"]
    out = torch.full((N, d, C), float("nan"), device=dev)
    z = torch.full((N, d, C), float("nan"), device=dev)
    perm = torch.full((E,), -1, dtype=torch.int32, device=dev)
    off = torch.full((N + 1,), -1, dtype=torch.int32, device=dev)
    got = tdn.forward_noalloc(*args, L=w["L"], r_cut=w["r_cut"], edges_sorted=w["presorted"], out=out, z=z,
                              perm=perm, offsets=off)
    torch.cuda.synchronize()
    return ref, got


def _check(w, A, B, D, ref, got):
    assert torch.equal(got.perm, ref.perm) and torch.equal(got.offsets, ref.offsets)
    assert torch.equal(got.out, ref.out)
    assert torch.equal(got.z, ref.z)
    oracle = layer.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], w["r_cut"],
                           w["L"])
    assert rel_err(got.out.cpu(), oracle) < TOL_F32
    check_rows(got.out.cpu(), oracle, TOL_F32, "out")


def test_noalloc_forward_equals_workspace_forward_on_consecutive_calls():
    # first call: the 960-node molecular workload (about 20 MiB of scratch)
    w1 = workloads.make_workload("molecules960_L3_C64_R64")
    A1, B1, D1 = load_factors(w1["L"], w1["R"])
    print(f"noalloc call 1: {w1['name']} N={w1['N']} E={w1['E']}", flush=True)
    ref1, got1 = _run_both(w1, A1, B1, D1)
    _check(w1, A1, B1, D1, ref1, got1)
    # second call, smaller and with unsorted edges (the sort's buffers come
    # from the same area); what the first call left there must not matter
    w2 = workloads.random_graph(41, n_nodes=50, n_edges=700, L=3, C=48, R=40, sort=False)
    A2, B2, D2 = random_factors(3, 40, 41)
    print(f"noalloc call 2: random N={w2['N']} E={w2['E']}", flush=True)
    ref2, got2 = _run_both(w2, A2, B2, D2)
    _check(w2, A2, B2, D2, ref2, got2)


def test_noalloc_rejects_problems_beyond_its_scratch():
    # the 3200-node headline size needs about 116 MiB: rejected on the host
    # before any launch, with the outputs left as they were
    w = workloads.make_workload("molecules3200_L4_C128_R128")
    A, B, D = load_factors(w["L"], w["R"])
    dev = "cuda"
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    N, d, C, E = w["N"], w["d"], w["C"], w["E"]
    out = torch.zeros((N, d, C), device=dev)
    perm = torch.zeros((E,), dtype=torch.int32, device=dev)
    off = torch.zeros((N + 1,), dtype=torch.int32, device=dev)
    with pytest.raises(tdn.TdnError, match="TDN_ERR_SCRATCH_LIMIT"):
        tdn.forward_noalloc(t(w["x"]), t(w["edge_vec"]), t(w["edge_index"]), t(A), t(B), t(D), t(w["W"]),
                            t(w["radial_w"]), L=w["L"], r_cut=w["r_cut"], edges_sorted=True, out=out, perm=perm,
                            offsets=off)
    torch.cuda.synchronize()
    assert not torch.any(out) and not torch.any(perm) and not torch.any(off)
