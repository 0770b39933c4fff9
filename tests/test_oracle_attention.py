"""Pins of the attention block's oracle (oracle/attention.py): with constant
logits it is the CP layer of oracle/layer.py divided by the in-degree (mean
aggregation); its weights are positive and sum to one over each destination's
edges per head; two edges into one node reproduce the logistic function of
their logit difference (hand-computed logits); with Thm. 2's exact per-path
factors it is rotation equivariant;
identical heads equal one head; it does not depend on the order of the edges;
and each head scales its own channel block."""
import numpy as np
import pytest
from scipy.special import expit

import workloads
from oracle import attention, cg_tensor, dense_layer, layer, wigner


def _graph(seed, L=2, N=14, E=120, C=8, R=6):
    return workloads.random_graph(seed, n_nodes=N, n_edges=E, L=L, C=C, R=R)


def _factors(L, R, seed):
    rng = np.random.default_rng(seed)
    d = (L + 1) ** 2
    return [rng.standard_normal((d, R)) / np.sqrt(d) for _ in range(3)]


def _att_weights(C, n_radial, F, H, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    W1 = scale * rng.standard_normal((2 * C + n_radial, F)) / np.sqrt(2 * C + n_radial)
    w2 = scale * rng.standard_normal((F, H)) / np.sqrt(F)
    return W1, w2


def _fwd(w, A, B, D, W1, w2, **kw):
    return attention.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], W1, w2,
                             w["r_cut"], w["L"], **kw)


@pytest.mark.parametrize("H", [1, 2, 4])
def test_constant_logits_give_the_mean_of_the_cp_messages(H):
    w = _graph(1)
    A, B, D = _factors(2, 6, 1)
    W1 = np.zeros((2 * w["C"] + w["n_radial"], 5))
    w2 = np.zeros((5, H))
    out, alpha = _fwd(w, A, B, D, W1, w2)
    deg = np.bincount(w["edge_index"][1], minlength=w["N"]).astype(np.float64)
    want = layer.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], w["r_cut"], 2)
    want = want / np.maximum(deg, 1)[:, None, None]
    np.testing.assert_allclose(out, want, rtol=1e-12, atol=1e-12 * np.max(np.abs(want)))
    np.testing.assert_allclose(alpha, 1.0 / deg[w["edge_index"][1]][:, None] * np.ones((1, H)), rtol=1e-14)


def test_weights_positive_and_normalised_per_destination_and_head():
    w = _graph(2, N=20, E=150)
    A, B, D = _factors(2, 6, 2)
    W1, w2 = _att_weights(w["C"], w["n_radial"], 7, 4, 2, scale=3.0)
    out, alpha = _fwd(w, A, B, D, W1, w2)
    assert np.all(alpha > 0)
    s = np.zeros((w["N"], 4))
    np.add.at(s, w["edge_index"][1], alpha)
    has = np.bincount(w["edge_index"][1], minlength=w["N"]) > 0
    np.testing.assert_allclose(s[has], 1.0, rtol=1e-13)
    assert np.all(out[~has] == 0)


def test_two_edges_follow_the_logistic_function_of_the_logit_difference():
    # one destination, two edges, one head, one hidden unit reading channel 0
    # of the source's degree-0 row: a_e = LeakyReLU(x[s_e]^(0)[0]) with x
    # values 2 and -1, so a = (2, -0.2) and alpha_1 = 1 / (1 + exp(-2.2))
    L, C = 1, 2
    w = workloads.random_graph(3, n_nodes=3, n_edges=2, L=L, C=C, R=4)
    w["edge_index"] = np.array([[1, 2], [0, 0]], np.int32)
    x = np.asarray(w["x"], np.float64).copy()
    x[1, 0, 0], x[2, 0, 0] = 2.0, -1.0
    w["x"] = x
    W1 = np.zeros((2 * C + w["n_radial"], 1))
    W1[C + 0, 0] = 1.0                       # rows C.. 2C-1 read x[s]^(0)
    w2 = np.ones((1, 1))
    A, B, D = _factors(L, 4, 3)
    _, alpha = _fwd(w, A, B, D, W1, w2)
    np.testing.assert_allclose(alpha[:, 0], [expit(2.2), expit(-2.2)], rtol=1e-14)


@pytest.mark.parametrize("L", [1, 2])
def test_rotation_equivariance(L):
    # exact per-path factors (Thm. 2) with one radial weight per path make the
    # messages equivariant; the logits see only invariants
    D, A, B, rank_path = dense_layer.exact_cp_factors(L)
    P = len(cg_tensor.paths(L))
    w = _graph(10 + L, L=L, C=8, R=P)
    w["radial_w"] = np.asarray(w["radial_w"], np.float64)[:, rank_path]
    W1, w2 = _att_weights(w["C"], w["n_radial"], 6, 2, 10 + L, scale=2.0)
    Rm = wigner.random_rotation(np.random.default_rng(L))
    Dr = wigner.wigner_d_full(L, Rm)
    out, alpha = _fwd(w, A, B, D, W1, w2)
    w2x = dict(w)
    w2x["x"] = np.einsum("ab,nbc->nac", Dr, np.asarray(w["x"], np.float64))
    w2x["edge_vec"] = np.asarray(w["edge_vec"], np.float64) @ Rm.T
    out2, alpha2 = _fwd(w2x, A, B, D, W1, w2)
    np.testing.assert_allclose(alpha2, alpha, rtol=1e-12)
    np.testing.assert_allclose(out2, np.einsum("ab,nbc->nac", Dr, out), rtol=0, atol=1e-10 * np.max(np.abs(out)))


def test_identical_heads_equal_one_head():
    w = _graph(4)
    A, B, D = _factors(2, 6, 4)
    W1, w2 = _att_weights(w["C"], w["n_radial"], 5, 1, 4, scale=2.0)
    out1, _ = _fwd(w, A, B, D, W1, w2)
    out4, alpha4 = _fwd(w, A, B, D, W1, np.repeat(w2, 4, axis=1))
    np.testing.assert_allclose(out4, out1, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(alpha4[:, 1:], alpha4[:, :1].repeat(3, axis=1), rtol=1e-15)


def test_independent_of_the_edge_order():
    w = _graph(5, N=10, E=90)
    A, B, D = _factors(2, 6, 5)
    W1, w2 = _att_weights(w["C"], w["n_radial"], 6, 2, 5, scale=2.0)
    out, alpha = _fwd(w, A, B, D, W1, w2)
    p = np.random.default_rng(0).permutation(w["E"])
    w2x = dict(w)
    w2x["edge_index"] = w["edge_index"][:, p]
    w2x["edge_vec"] = w["edge_vec"][p]
    outp, alphap = _fwd(w2x, A, B, D, W1, w2)
    np.testing.assert_allclose(outp, out, rtol=1e-12, atol=1e-13 * np.max(np.abs(out)))
    np.testing.assert_allclose(alphap, alpha[p], rtol=1e-13)


def test_each_head_scales_its_own_channel_block():
    # two heads over C = 8 channels: head 0 constant logits (the mean), head 1
    # not; with W = I the first four output channels are the mean of the
    # messages and the last four are not
    w = _graph(6)
    w["W"] = np.eye(w["C"])
    A, B, D = _factors(2, 6, 6)
    W1, w2 = _att_weights(w["C"], w["n_radial"], 5, 2, 6, scale=3.0)
    w2[:, 0] = 0.0
    out, alpha = _fwd(w, A, B, D, W1, w2)
    deg = np.bincount(w["edge_index"][1], minlength=w["N"]).astype(np.float64)
    mean = layer.forward(w["x"], w["edge_index"], w["edge_vec"], A, B, D, w["W"], w["radial_w"], w["r_cut"], 2)
    mean = mean / np.maximum(deg, 1)[:, None, None]
    np.testing.assert_allclose(out[:, :, :4], mean[:, :, :4], rtol=1e-12, atol=1e-13 * np.max(np.abs(mean)))
    assert np.max(np.abs(out[:, :, 4:] - mean[:, :, 4:])) > 1e-3 * np.max(np.abs(mean))
