"""Host-side tests of the C ABI that need no GPU: the library loads, exports
every entry point that include/tdn.h declares, and rejects bad arguments
before touching any device."""
import ctypes
import os
import re

import pytest

import paper_2507_01131_amd as tdn

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "tdn.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tdn_[a-z_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    syms = declared_symbols()
    assert len(syms) >= 10
    L = tdn.lib()
    for s in syms:
        assert hasattr(L, s), s


def _problem(**kw):
    base = dict(L=4, C=128, R=128, n_nodes=100, n_edges=1000, r_cut=6.0)
    base.update(kw)
    return tdn.make_problem(**base)


FAKE = ctypes.c_void_p(0x1000)   # never dereferenced: every case returns before any launch


def _fwd(p, ws_bytes=1 << 40, **override):
    args = dict(x=FAKE, vec=FAKE, ei=FAKE, A=FAKE, B=FAKE, D=FAKE, W=FAKE, rw=FAKE, out=FAKE, z=None, perm=FAKE,
                off=FAKE, ws=FAKE)
    args.update(override)
    return tdn.lib().tdn_cp_tp_forward(None if p is None else ctypes.byref(p), args["x"], args["vec"], args["ei"],
                                       args["A"], args["B"], args["D"], args["W"], args["rw"], args["out"], args["z"],
                                       args["perm"], args["off"], args["ws"], ws_bytes, None)


def _bwd(p, ws_bytes=1 << 40, **override):
    args = dict(x=FAKE, vec=FAKE, ei=FAKE, A=FAKE, B=FAKE, D=FAKE, W=FAKE, rw=FAKE, perm=FAKE, off=FAKE, z=None,
                g=FAKE, gx=FAKE, gW=FAKE, gv=FAKE, gr=FAKE, ws=FAKE)
    args.update(override)
    return tdn.lib().tdn_cp_tp_backward(ctypes.byref(p), args["x"], args["vec"], args["ei"], args["A"], args["B"],
                                        args["D"], args["W"], args["rw"], args["perm"], args["off"], args["z"],
                                        args["g"], args["gx"], args["gW"], args["gv"], args["gr"], args["ws"],
                                        ws_bytes, None)


@pytest.mark.parametrize("kw,status", [
    (dict(L=7), 2), (dict(L=-1), 2), (dict(C=8), 2), (dict(C=100), 2), (dict(C=512), 2), (dict(R=0), 2),
    (dict(R=4097), 2), (dict(n_nodes=-1), 2), (dict(n_edges=-5), 2), (dict(n_nodes=0, n_edges=3), 2),
    (dict(n_radial=1), 2), (dict(r_cut=0.0), 2), (dict(r_cut=float("nan")), 2), (dict(feat_dtype=7), 3),
])
def test_bad_problem_is_rejected(kw, status):
    p = _problem(**kw)
    assert _fwd(p) == status
    assert _bwd(p) == status
    f, b = ctypes.c_size_t(), ctypes.c_size_t()
    assert tdn.lib().tdn_workspace_size(ctypes.byref(p), ctypes.byref(f), ctypes.byref(b)) == status


def test_null_problem_and_pointers():
    assert _fwd(None) == 1
    p = _problem()
    for k in ["x", "vec", "ei", "A", "B", "D", "W", "rw", "out", "perm", "off", "ws"]:
        assert _fwd(p, **{k: None}) == 1, k
    for k in ["x", "vec", "ei", "A", "B", "D", "W", "rw", "perm", "off", "g", "ws"]:
        assert _bwd(p, **{k: None}) == 1, k


def test_edge_arrays_optional_without_edges():
    # E = 0: edge pointers may be NULL; the call then proceeds to the device
    # check, which fails on a machine without a GPU (status 8 or 9), never 1.
    p = _problem(n_edges=0)
    assert _fwd(p, ws_bytes=0, vec=None, ei=None, perm=None) == 4
    f, _ = tdn.workspace_size(p)
    assert f > 0


def test_workspace_too_small():
    p = _problem()
    f, b = tdn.workspace_size(p)
    assert _fwd(p, ws_bytes=f - 1) == 4
    assert _bwd(p, ws_bytes=b - 1) == 4
    # the saved-activation buffer dominates: N*d*C floats
    assert f >= 100 * 25 * 128 * 4
    assert b >= 2 * 100 * 25 * 128 * 4


def test_sort_and_sh_argument_checks():
    L = tdn.lib()
    nb = ctypes.c_size_t()
    assert L.tdn_sort_workspace_size(-1, 5, ctypes.byref(nb)) == 2
    assert L.tdn_sort_workspace_size(0, 5, ctypes.byref(nb)) == 2
    assert L.tdn_sort_workspace_size(10, 5, None) == 1
    assert L.tdn_sort_workspace_size(10, 5, ctypes.byref(nb)) == 0 and nb.value > 0
    assert L.tdn_sort_by_key(10, 5, FAKE, FAKE, FAKE, FAKE, 1, None) == 4
    assert L.tdn_sort_by_key(10, 5, None, FAKE, FAKE, FAKE, 1 << 30, None) == 1
    assert L.tdn_spherical_harmonics(7, 5, FAKE, FAKE, None, None) == 2
    assert L.tdn_spherical_harmonics(3, 5, None, FAKE, None, None) == 1


def _gp(N=100, G=2, r_cut=5.0, cap=0, per=(0, 0, 0)):
    return tdn.GraphProblem(N, G, r_cut, cap, (ctypes.c_int32 * 3)(*per))


def _rg(g, ws_bytes=1 << 40, capacity=0, **override):
    args = dict(pos=FAKE, ptr=FAKE, cell=None, ei=None, ev=None, im=None, off=None, ws=FAKE)
    args.update(override)
    n = ctypes.c_int64(-1)
    st = tdn.lib().tdn_radius_graph(None if g is None else ctypes.byref(g), args["pos"], args["ptr"], args["cell"],
                                    capacity, args["ei"], args["ev"], args["im"], args["off"], ctypes.byref(n),
                                    args["ws"], ws_bytes, None)
    return st, n.value


@pytest.mark.parametrize("g,status", [
    (None, 1),
    (_gp(N=-1), 2), (_gp(N=1 << 26), 2), (_gp(G=0), 2), (_gp(r_cut=0.0), 2), (_gp(r_cut=float("nan")), 2),
    (_gp(cap=-1), 2), (_gp(per=(0, 2, 0)), 2),
])
def test_radius_graph_problem_checks(g, status):
    assert _rg(g)[0] == status
    if g is not None:
        nb = ctypes.c_size_t()
        assert tdn.lib().tdn_radius_graph_workspace_size(ctypes.byref(g), ctypes.byref(nb)) == status


def test_radius_graph_argument_checks():
    L = tdn.lib()
    nb = ctypes.c_size_t()
    assert L.tdn_radius_graph_workspace_size(ctypes.byref(_gp()), None) == 1
    assert L.tdn_radius_graph_workspace_size(ctypes.byref(_gp()), ctypes.byref(nb)) == 0 and nb.value > 0
    assert _rg(_gp(), pos=None)[0] == 1
    assert _rg(_gp(), ptr=None)[0] == 1
    assert _rg(_gp(), ws=None)[0] == 1
    assert _rg(_gp(per=(1, 0, 0)))[0] == 1                    # periodic needs cell
    assert _rg(_gp(), capacity=-5)[0] == 2
    assert _rg(_gp(), capacity=10)[0] == 1                    # capacity without buffers
    assert _rg(_gp(), capacity=10, ei=FAKE)[0] == 1
    assert _rg(_gp(), ws_bytes=nb.value - 1)[0] == 4


def test_status_strings():
    for s in range(14):
        assert tdn.status_string(s) not in ("", "unknown status")
    assert tdn.status_string(0) == "ok"


def test_timer_bookkeeping_without_launches():
    tdn.timer_enable(True)
    ms, n = tdn.timer_read("cp_edge_fwd")
    assert ms == 0.0 and n == 0
    tdn.timer_enable(False)


def _dense(p, ws_bytes=1 << 40, nnz=100, **override):
    args = dict(x=FAKE, vec=FAKE, ei=FAKE, row=FAKE, col=FAKE, val=FAKE, pw=FAKE, W=FAKE, out=FAKE, z=None,
                perm=FAKE, off=FAKE, ws=FAKE)
    args.update(override)
    return tdn.lib().tdn_dense_tp_forward(None if p is None else ctypes.byref(p), args["x"], args["vec"], args["ei"],
                                          args["row"], args["col"], args["val"], nnz, args["pw"], args["W"],
                                          args["out"], args["z"], args["perm"], args["off"], args["ws"], ws_bytes,
                                          None)


@pytest.mark.parametrize("L,n_path", [(0, 1), (1, 5), (2, 15), (3, 34), (4, 65), (5, 111), (6, 175)])
def test_dense_forward_argument_checks(L, n_path):
    # R must be the number of paths of degree L (Sec. 2: l1, l2 <= L,
    # |l1 - l2| <= l3 <= min(l1 + l2, L))
    good = _problem(L=L, R=n_path)
    assert _dense(good, ws_bytes=0) == 4                       # everything else accepted
    assert _dense(_problem(L=L, R=n_path + 1)) == 2
    assert _dense(_problem(L=L, R=n_path, feat_dtype=tdn.TDN_BF16)) == 3
    assert _dense(good, nnz=-1) == 2
    assert _dense(None) == 1
    for k in ["x", "vec", "ei", "row", "col", "val", "pw", "W", "out", "perm", "off", "ws"]:
        assert _dense(good, **{k: None}) == 1, k
    assert _dense(good, ws_bytes=0, nnz=0, col=None, val=None) == 4   # an empty table needs no entries


def _dense_un(p, ws_bytes=1 << 40, nnz=100, **override):
    args = dict(x=FAKE, vec=FAKE, ei=FAKE, row=FAKE, col=FAKE, val=FAKE, pw=FAKE, Wp=FAKE, out=FAKE,
                perm=FAKE, off=FAKE, ws=FAKE)
    args.update(override)
    return tdn.lib().tdn_dense_tp_forward_unshared(None if p is None else ctypes.byref(p), args["x"], args["vec"],
                                                   args["ei"], args["row"], args["col"], args["val"], nnz,
                                                   args["pw"], args["Wp"], args["out"], args["perm"], args["off"],
                                                   args["ws"], ws_bytes, None)


@pytest.mark.parametrize("L,n_path,n_rows", [(0, 1, 1), (1, 5, 11), (2, 15, 51), (3, 34, 156), (4, 65, 375),
                                             (5, 111, 771), (6, 175, 1421)])
def test_dense_unshared_argument_checks_and_workspace(L, n_path, n_rows):
    # the per-path node sums take sum over paths of (2 l3 + 1) rows per node
    assert n_rows == sum(2 * l3 + 1 for l1 in range(L + 1) for l2 in range(L + 1)
                         for l3 in range(abs(l1 - l2), min(l1 + l2, L) + 1))
    good = _problem(L=L, R=n_path, C=96)
    fwd, _ = tdn.workspace_size(good)
    un = ctypes.c_size_t(0)
    assert tdn.lib().tdn_dense_tp_unshared_workspace_size(ctypes.byref(good), ctypes.byref(un)) == 0
    assert un.value >= fwd + 100 * n_rows * 96 * 4
    assert un.value < fwd + 100 * n_rows * 96 * 4 + 4096
    assert tdn.lib().tdn_dense_tp_unshared_workspace_size(ctypes.byref(good), None) == 1
    assert _dense_un(good, ws_bytes=un.value - 1) == 4
    assert _dense_un(good, ws_bytes=0) == 4
    assert _dense_un(_problem(L=L, R=n_path + 1)) == 2
    assert _dense_un(_problem(L=L, R=n_path, C=144)) == 2             # C <= 128
    assert _dense_un(_problem(L=L, R=n_path, feat_dtype=tdn.TDN_BF16)) == 3
    assert _dense_un(good, nnz=-1) == 2
    assert _dense_un(None) == 1
    for k in ["x", "vec", "ei", "row", "col", "val", "pw", "Wp", "out", "perm", "off", "ws"]:
        assert _dense_un(good, **{k: None}) == 1, k
    assert _dense_un(good, ws_bytes=0, nnz=0, col=None, val=None) == 4


def _tp3(p, ws_bytes=1 << 40, **override):
    args = dict(x=FAKE, vec=FAKE, ei=FAKE, A=FAKE, A2=FAKE, B=FAKE, D=FAKE, W=FAKE, rw=FAKE, out=FAKE, z=None,
                perm=FAKE, off=FAKE, ws=FAKE)
    args.update(override)
    return tdn.lib().tdn_cp_tp3_forward(None if p is None else ctypes.byref(p), args["x"], args["vec"], args["ei"],
                                        args["A"], args["A2"], args["B"], args["D"], args["W"], args["rw"],
                                        args["out"], args["z"], args["perm"], args["off"], args["ws"], ws_bytes, None)


def test_three_input_forward_argument_checks():
    good = _problem(L=4)
    assert _tp3(good, ws_bytes=0) == 4
    assert _tp3(_problem(L=1)) == 2 and _tp3(_problem(L=5)) == 2      # 2 <= L <= 4
    assert _tp3(_problem(feat_dtype=tdn.TDN_BF16)) == 3
    assert _tp3(None) == 1
    for k in ["x", "vec", "ei", "A", "A2", "B", "D", "W", "rw", "out", "perm", "off", "ws"]:
        assert _tp3(good, **{k: None}) == 1, k
    # the workspace covers the three-input product's edge ranges too
    f, _ = tdn.workspace_size(good)
    assert _tp3(good, ws_bytes=f - 1) == 4


def test_ps_linear_argument_checks():
    L = tdn.lib()
    nb = ctypes.c_size_t()
    assert L.tdn_ps_linear_workspace_size(128, tdn.TDN_F32, ctypes.byref(nb)) == 0 and nb.value > 0
    assert L.tdn_ps_linear_workspace_size(128, tdn.TDN_BF16, ctypes.byref(nb)) == 0 and nb.value == 0
    assert L.tdn_ps_linear_workspace_size(100, tdn.TDN_F32, ctypes.byref(nb)) == 2
    assert L.tdn_ps_linear_workspace_size(128, 9, ctypes.byref(nb)) == 3
    assert L.tdn_ps_linear(10, 2, 64, FAKE, FAKE, 9, FAKE, FAKE, 1 << 30, None) == 3
    assert L.tdn_ps_linear(10, 7, 64, FAKE, FAKE, tdn.TDN_F32, FAKE, FAKE, 1 << 30, None) == 2
    assert L.tdn_ps_linear(10, 2, 40, FAKE, FAKE, tdn.TDN_F32, FAKE, FAKE, 1 << 30, None) == 2
    assert L.tdn_ps_linear(-1, 2, 64, FAKE, FAKE, tdn.TDN_F32, FAKE, FAKE, 1 << 30, None) == 2
    assert L.tdn_ps_linear(10, 2, 64, None, FAKE, tdn.TDN_F32, FAKE, FAKE, 1 << 30, None) == 1
    assert L.tdn_ps_linear(10, 2, 64, FAKE, None, tdn.TDN_F32, FAKE, FAKE, 1 << 30, None) == 1
    assert L.tdn_ps_linear(10, 2, 64, FAKE, FAKE, tdn.TDN_F32, FAKE, None, 1 << 30, None) == 1
    assert L.tdn_ps_linear(10, 2, 64, FAKE, FAKE, tdn.TDN_F32, FAKE, FAKE, 0, None) == 4


def test_noalloc_forward_rejects_problems_beyond_its_scratch():
    # a host-side check made before any device work: the headline size needs
    # more than the fixed scratch area holds
    L = tdn.lib()
    p = tdn.make_problem(4, 128, 128, 3200, 151118, 6.0)
    f, _ = tdn.workspace_size(p)
    assert f > tdn.NOALLOC_SCRATCH_BYTES
    st = L.tdn_cp_tp_forward_noalloc(ctypes.byref(p), *([None] * 12), None)
    assert st == 13 and tdn.STATUS[st] == "TDN_ERR_SCRATCH_LIMIT"
    bad = tdn.make_problem(4, 100, 128, 10, 10, 6.0)     # C not a multiple of 16
    assert L.tdn_cp_tp_forward_noalloc(ctypes.byref(bad), *([None] * 12), None) == 2


def _abl(p, variant, ws_bytes=1 << 40, **override):
    args = dict(x=FAKE, vec=FAKE, ei=FAKE, A=FAKE, B=FAKE, D=FAKE, W=FAKE, rw=FAKE, out=FAKE, z=None, perm=FAKE,
                off=FAKE, ws=FAKE)
    args.update(override)
    return tdn.lib().tdn_ablation_forward(None if p is None else ctypes.byref(p), variant, args["x"], args["vec"],
                                          args["ei"], args["A"], args["B"], args["D"], args["W"], args["rw"],
                                          args["out"], args["z"], args["perm"], args["off"], args["ws"], ws_bytes,
                                          None)


@pytest.mark.parametrize("variant", [tdn.ABL_FACTORS_GLOBAL, tdn.ABL_Y_TABLE, tdn.ABL_VALU])
def test_ablation_forward_argument_checks(variant):
    good = _problem(L=4, C=128, R=128)
    need = ctypes.c_size_t(0)
    assert tdn.lib().tdn_ablation_workspace_size(ctypes.byref(good), variant, ctypes.byref(need)) == 0
    fwd, _ = tdn.workspace_size(good)
    assert need.value >= fwd
    if variant == tdn.ABL_Y_TABLE:      # one row of d harmonics per edge
        assert need.value >= fwd + 1000 * 25 * 4
    assert _abl(good, variant, ws_bytes=need.value - 1) == 4
    assert _abl(good, 0) == 2 and _abl(good, 4) == 2
    assert _abl(_problem(L=1, R=32), variant) == 2
    assert _abl(_problem(L=5, R=32), variant) == 2
    assert _abl(_problem(L=4, R=300), variant) == 2
    assert _abl(_problem(L=4, feat_dtype=tdn.TDN_BF16), variant) == 3
    if variant == tdn.ABL_VALU:
        assert _abl(_problem(L=4, C=160), variant) == 2   # R, C <= 128
    assert _abl(None, variant) == 1
    for k in ["x", "vec", "ei", "A", "B", "D", "W", "rw", "out", "perm", "off", "ws"]:
        assert _abl(good, variant, **{k: None}) == 1, k


def _att(p, H=2, F=8, ws_bytes=1 << 40, **override):
    args = dict(x=FAKE, vec=FAKE, ei=FAKE, A=FAKE, B=FAKE, D=FAKE, W=FAKE, rw=FAKE, w1=FAKE, w2=FAKE, out=FAKE,
                alpha=None, z=None, perm=FAKE, off=FAKE, ws=FAKE)
    args.update(override)
    return tdn.lib().tdn_attention_forward(None if p is None else ctypes.byref(p), H, F, args["x"], args["vec"],
                                           args["ei"], args["A"], args["B"], args["D"], args["W"], args["rw"],
                                           args["w1"], args["w2"], args["out"], args["alpha"], args["z"],
                                           args["perm"], args["off"], args["ws"], ws_bytes, None)


def test_attention_forward_argument_checks():
    good = _problem(L=4, C=128, R=128)
    need = ctypes.c_size_t(0)
    assert tdn.lib().tdn_attention_workspace_size(ctypes.byref(good), 4, 32, ctypes.byref(need)) == 0
    fwd, _ = tdn.workspace_size(good)
    assert need.value >= fwd + 2 * 100 * 32 * 4 + 1000 * 4 * 4       # Pt, Ps and the sorted weights
    assert _att(good, H=4, F=32, ws_bytes=need.value - 1) == 4
    assert _att(good, H=3) == 2                 # C not a multiple of 32 H
    assert _att(good, H=0) == 2 and _att(good, H=16) == 2
    assert _att(good, F=0) == 2 and _att(good, F=65) == 2
    assert _att(_problem(L=0, R=32)) == 2 and _att(_problem(L=5, R=32)) == 2
    assert _att(_problem(L=4, R=300)) == 2
    assert _att(_problem(L=4, feat_dtype=tdn.TDN_BF16)) == 3
    assert _att(None) == 1
    for k in ["x", "vec", "ei", "A", "B", "D", "W", "rw", "w1", "w2", "out", "perm", "off", "ws"]:
        assert _att(good, **{k: None}) == 1, k
