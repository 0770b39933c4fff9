"""GPU parity on inputs of wide dynamic range, through the C ABI.

The float32 path runs its 16-bit MFMA contractions on two-part fp16 splits of
operands scaled by one power of two per node row (or segment, tile or
factor).  These tests give every node row values spread over 2^-20 .. 2^20
across its degree rows and channels, make one node 2^40 times larger than
every other, and spread the output cotangent the same way (without the large
node, which keeps every product inside the float32 range), so that an operand
scaled or split with the wrong granularity loses the small values a row or a
segment holds.  Forward output, the saved Z and grad_x are checked per node
row, grad_edge_vec per edge against its magnitude scale, grad_W and the
radial-weight gradient elementwise against their largest value, all against
the float64 oracle at the float32 tolerance."""
import numpy as np
import pytest
import torch

import paper_2507_01131_amd as tdn
import workloads
from oracle import layer
from tests._gpu_helpers import (TOL_F32, check_elementwise, check_rows, check_scaled, grad_vec_scale, rel_err,
                                random_factors)

pytestmark = pytest.mark.gpu


def _spread(rng, shape, lo=-20, hi=20):
    """Per (node, degree row, channel) powers of two 2^(a[n, c] + b[n, k]) with
    a in [-12, 12] and b in [-8, 8], every node row reaching both ends."""
    N, d, C = shape
    a = rng.integers(-12, 13, size=(N, 1, C))
    b = rng.integers(-8, 9, size=(N, d, 1))
    a[:, 0, 0], a[:, 0, C - 1] = -12, 12
    b[:, 0, 0], b[:, d - 1, 0] = -8, 8
    e = a + b
    assert e.min() == lo and e.max() == hi
    return np.ldexp(np.float32(1.0), e).astype(np.float32)


def _wide_problem(seed, N, E, L, C, R, big=True):
    w = workloads.random_graph(seed, n_nodes=N, n_edges=E, L=L, C=C, R=R, sort=False)
    rng = np.random.default_rng(seed + 500)
    x = w["x"] * _spread(rng, w["x"].shape)
    G = w["grad_out"] * _spread(rng, w["grad_out"].shape)
    if big:
        # the node with most outgoing edges, 2^40 times every other row
        hub = int(np.argmax(np.bincount(w["edge_index"][0], minlength=N)))
        x[hub] *= np.float32(2.0 ** 40)
    w["x"], w["grad_out"] = x.astype(np.float32), G.astype(np.float32)
    return w


CASES = [
    dict(seed=31, N=60, E=1500, L=3, C=64, R=64),
    dict(seed=32, N=70, E=2000, L=4, C=128, R=128),
    dict(seed=33, N=40, E=900, L=2, C=48, R=40),
    dict(seed=34, N=40, E=800, L=6, C=64, R=64),
    dict(seed=35, N=30, E=600, L=5, C=96, R=100),
]


@pytest.mark.parametrize("cfg", CASES, ids=lambda c: f"L{c['L']}C{c['C']}R{c['R']}")
def test_wide_dynamic_range_forward_and_backward(cfg):
    c = dict(cfg)
    seed = c.pop("seed")
    w = _wide_problem(seed, **c)
    A, B, D = random_factors(w["L"], w["R"], seed)
    dev = "cuda"
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    res = tdn.forward(t(w["x"]), t(w["edge_vec"]), t(w["edge_index"]), t(A), t(B), t(D), t(w["W"]),
                      t(w["radial_w"]), L=w["L"], r_cut=w["r_cut"], edges_sorted=False)
    gx, gW, gv, gr = tdn.backward(res, t(w["grad_out"]), need_radial=True)
    torch.cuda.synchronize()
    args = (w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], w["r_cut"], w["L"])
    ref, zref = layer.forward(*args, return_z=True)
    rx, rW, rv, rr = layer.backward(*args, w["grad_out"], return_radial=True)
    out, z = res.out.cpu().numpy(), res.z.cpu().numpy()
    assert rel_err(out, ref) < TOL_F32
    check_rows(out, ref, TOL_F32, "out")
    check_rows(z, zref, TOL_F32, "z")
    check_rows(gx.cpu().numpy(), rx, TOL_F32, "grad_x")
    check_scaled(gv.cpu().numpy(), rv, grad_vec_scale(w, A, B, D), TOL_F32, "grad_edge_vec")
    assert rel_err(gv.cpu(), rv) < TOL_F32
    assert rel_err(gW.cpu(), rW) < TOL_F32
    check_elementwise(gW.cpu().numpy(), rW, TOL_F32, "grad_W")
    check_elementwise(gr.cpu().numpy(), rr, TOL_F32, "grad_radial_w")
