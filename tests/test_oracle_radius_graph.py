"""Pins of the radius-graph oracle (oracle/radius_graph.py) against lattice
geometry, symmetry, scalar brute force and the float64 builder that makes
the workload fixtures."""
import itertools

import numpy as np
import pytest

import workloads
from oracle import radius_graph as rg
from workloads import geometry


def _lattice(basis, a, reps):
    cells = np.array(list(itertools.product(range(reps), repeat=3)), dtype=np.float64)
    return ((cells[:, None, :] + np.asarray(basis)[None]) * a).reshape(-1, 3)


SC = [[0, 0, 0]]
FCC = [[0, 0, 0], [0.5, 0.5, 0], [0.5, 0, 0.5], [0, 0.5, 0.5]]


@pytest.mark.parametrize("basis,a,reps,r_cut,shells", [
    (SC, 2.0, 4, 2.5, {4.0: 6}),                           # simple cubic: 6 at a
    (SC, 2.0, 4, 3.0, {4.0: 6, 8.0: 12}),                  # + 12 at a*sqrt(2)
    (SC, 2.0, 4, 3.5, {4.0: 6, 8.0: 12, 12.0: 8}),         # + 8 at a*sqrt(3)
    (FCC, 3.6, 3, 3.0, {6.48: 12}),                        # fcc: 12 at a/sqrt(2)
    (FCC, 3.6, 3, 4.0, {6.48: 12, 12.96: 6}),              # + 6 at a
])
def test_periodic_lattices_have_their_coordination_shells(basis, a, reps, r_cut, shells):
    pos = _lattice(basis, a, reps).astype(np.float32)
    L = np.float32(a * reps)
    s, d, n, v = rg.radius_graph(pos, [0, len(pos)], [[L, L, L]], (True, True, True), r_cut)
    counts = np.bincount(d, minlength=len(pos))
    assert np.all(counts == sum(shells.values()))
    r2 = np.round(np.einsum("ij,ij->i", v.astype(np.float64), v), 2)
    for sq, k in shells.items():
        assert np.sum(r2 == round(sq, 2)) == k * len(pos)


def test_box_between_one_and_two_cutoffs_joins_a_pair_through_two_images():
    # x periodic with L = 3, atoms 1.5 apart: both the direct vector and the
    # one through the neighbouring box (length 1.5 each) are within 2.9;
    # an atom's own images lie exactly L = 3 away and never qualify
    pos = np.array([[0.5, 0.0, 0.0], [2.0, 0.0, 0.0]], np.float32)
    cell = [[3.0, 0.0, 0.0]]
    s, d, n, v = rg.radius_graph(pos, [0, 2], cell, (True, False, False), 2.9)
    got = [(int(a), int(b), int(c[0]), float(x[0])) for a, b, c, x in zip(s, d, n, v)]
    assert got == [(1, 0, -1, -1.5), (1, 0, 0, 1.5), (0, 1, 0, -1.5), (0, 1, 1, 1.5)]
    s, d, n, v = rg.radius_graph(pos, [0, 2], cell, (True, False, False), 3.0)
    assert len(s) == 4                                    # |r| = 3 is not < 3
    s, d, n, v = rg.radius_graph(pos, [0, 2], cell, (True, False, False), 1.5)
    assert len(s) == 0                                    # strict cutoff


def test_reversed_edges_exist_with_exactly_negated_vectors():
    rng = np.random.default_rng(3)
    L = np.float32(9.0)
    pos = rng.uniform(0, L, size=(150, 3)).astype(np.float32)
    s, d, n, v = rg.radius_graph(pos, [0, 150], [[L, L, 0]], (True, True, False), 2.7)
    fwd = {(a, b, tuple(c)): tuple(x) for a, b, c, x in zip(s, d, n, v)}
    assert len(fwd) == len(s) > 500
    for (a, b, c), x in fwd.items():
        y = fwd[(b, a, tuple(-np.asarray(c)))]
        assert tuple(-np.float32(t) for t in x) == y


def test_scalar_brute_force_on_a_tiny_batch():
    rng = np.random.default_rng(5)
    ptr = [0, 7, 7, 14]                       # an empty system in the middle
    L = np.float32(4.0)
    cell = np.array([[L, 0, 0]] * 3, np.float32)
    pos = rng.uniform(0, 4.0, size=(14, 3)).astype(np.float32)
    r_cut = 2.2
    rc2 = np.float32(r_cut) * np.float32(r_cut)
    want = []
    for g in range(3):
        for dst in range(ptr[g], ptr[g + 1]):
            for src in range(ptr[g], ptr[g + 1]):
                for nx in (-1, 0, 1):
                    if src == dst and nx == 0:
                        continue
                    r = [np.float32(pos[src, k] - pos[dst, k]) for k in range(3)]
                    r[0] = np.float32(r[0] + np.float32(nx) * L)
                    q = np.float32(np.float32(np.float32(r[0] * r[0]) + np.float32(r[1] * r[1]))
                                   + np.float32(r[2] * r[2]))
                    if q < rc2:
                        want.append((dst, src, nx, r[0], r[1], r[2]))
    want.sort(key=lambda t: (t[0], t[1], t[2]))
    s, d, n, v = rg.radius_graph(pos, ptr, cell, (True, False, False), r_cut)
    got = [(int(a), int(b), int(c[0]), x[0], x[1], x[2]) for b, a, c, x in zip(s, d, n, v)]
    assert got == want and len(want) > 10


@pytest.mark.parametrize("name,n_dst", [("cube64_L2_C16_R32", None), ("molecules960_L3_C64_R64", None),
                                        ("slabs4960_L6_C128_R256", 400), ("bulk4096_L4_C256_R128_bf16", 200)])
def test_matches_the_float64_fixture_builder_away_from_the_cutoff(name, n_dst):
    w = workloads.WORKLOADS[name]
    geo = workloads.graph_inputs(name)
    per, ptr, cell32, pos32 = geo["periodic"], geo["graph_ptr"], geo["cell"], geo["pos"]
    n_all, fs, fd, fv = workloads.make_graph(w)
    rng = np.random.default_rng(0)
    dsts = np.arange(n_all) if n_dst is None else np.sort(rng.choice(n_all, n_dst, replace=False))
    s, d, n, v = rg.radius_graph(pos32, ptr, cell32, per, geo["r_cut"], dst_nodes=dsts)
    mine = {(a, b): x for a, b, x in zip(s, d, v)}     # at most one image per pair here (boxes >= 2 r_cut)
    assert len(mine) == len(s)
    sel = np.isin(fd, dsts)
    theirs = {(a, b): x for a, b, x in zip(fs[sel], fd[sel], fv[sel])}
    for key in set(mine) ^ set(theirs):
        x = mine.get(key, theirs.get(key))
        assert abs(np.linalg.norm(np.asarray(x, np.float64)) - geo["r_cut"]) < 1e-4, key
    common = set(mine) & set(theirs)
    assert len(common) > 0.999 * max(len(mine), len(theirs))
    diff = max(np.max(np.abs(np.asarray(mine[k], np.float64) - theirs[k])) for k in common)
    assert diff < 1e-5


def test_neighbour_cap_keeps_the_nearest():
    rng = np.random.default_rng(7)
    L = np.float32(7.0)
    pos = rng.uniform(0, L, size=(120, 3)).astype(np.float32)
    args = (pos, [0, 120], [[L, L, L]], (True, True, True), 3.0)
    s, d, n, v = rg.radius_graph(*args)
    cs, cd, cn, cv = rg.radius_graph(*args, max_neighbors=8)
    full = np.bincount(d, minlength=120)
    assert np.all(np.bincount(cd, minlength=120) == np.minimum(full, 8)) and full.max() > 8
    for t in range(120):
        kept = np.einsum("ij,ij->i", cv[cd == t].astype(np.float64), cv[cd == t])
        allr = np.sort(np.einsum("ij,ij->i", v[d == t].astype(np.float64), v[d == t]))
        np.testing.assert_allclose(np.sort(kept), allr[:len(kept)], rtol=1e-6)
        order = list(zip(cs[cd == t], rg.image_code(cn[cd == t])))
        assert order == sorted(order)


def test_systems_do_not_connect_and_empty_inputs():
    rng = np.random.default_rng(9)
    one = rng.uniform(0, 5, size=(30, 3)).astype(np.float32)
    pos = np.concatenate([one, one])
    s, d, n, v = rg.radius_graph(pos, [0, 30, 60], None, (False, False, False), 2.5)
    a = (s < 30) & (d < 30)
    b = (s >= 30) & (d >= 30)
    assert np.all(a | b)
    np.testing.assert_array_equal(s[a] + 30, s[b])
    np.testing.assert_array_equal(v[a], v[b])
    s, d, n, v = rg.radius_graph(np.zeros((1, 3), np.float32), [0, 1], None, (False,) * 3, 2.0)
    assert len(s) == 0
    s, d, n, v = rg.radius_graph(np.zeros((0, 3), np.float32), [0], None, (False,) * 3, 2.0)
    assert len(s) == 0 and v.shape == (0, 3)


def test_host_builder_conventions_match():
    # the fixture builder's vector convention is the oracle's with n = 0
    pos = np.array([[0.0, 0, 0], [1.0, 0.5, 0]])
    s, t, v = geometry.radius_graph(pos, 2.0)
    assert list(zip(s, t)) == [(1, 0), (0, 1)]
    np.testing.assert_allclose(v[0], pos[1] - pos[0])
