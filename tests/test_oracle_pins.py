"""Pins of the CPU oracle to facts that do not come from the oracle itself:
hand-worked values, dense brute force (the fused Gather equals the
adjacency x embedding product, Sec. 3.2 / Fig. 7b), closed forms,
invariants (softmax weights sum to 1, permutation equivariance) and special
cases that reduce to textbook operations.  CPU only."""
import json
import math
import os

import numpy as np
import pytest

from helpers import dense_adjacency, edges_to_csr, rel_err, tiny_graphs
from oracle import saga_oracle as O

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def _graph(n, src, dst):
    rp, col, order = edges_to_csr(n, src, dst)
    return rp, col, order


# --------------------------------------------------------------------------
# hand-worked fixtures
# --------------------------------------------------------------------------
def test_gcn_hand_worked():
    g = _load("gcn_hand.json")
    src = [e[0] for e in g["edges_src_to_dst"]]
    dst = [e[1] for e in g["edges_src_to_dst"]]
    rp, col, _ = _graph(g["n"], src, dst)
    X = np.array(g["X"], dtype=np.float64)
    W = np.array(g["W"], dtype=np.float64)
    b = np.array(g["b"], dtype=np.float64)
    pre = O.gcn_layer(rp, col, X, W, b, "none")
    out = O.gcn_layer(rp, col, X, W, b, "relu")
    np.testing.assert_allclose(pre, g["pre_activation"], rtol=0, atol=1e-14)
    np.testing.assert_allclose(out, g["relu_output"], rtol=0, atol=1e-14)
    # transform-first association gives the same numbers
    out_tf = O.gcn_layer(rp, col, X, W, b, "relu", order="transform_first")
    np.testing.assert_allclose(out_tf, g["relu_output"], rtol=0, atol=1e-14)
    # the aggregate alone (identity transform)
    agg = O.gcn_layer(rp, col, X, np.eye(2), np.zeros(2), "none")
    np.testing.assert_allclose(agg, g["aggregate"], rtol=0, atol=1e-14)


def test_gat_hand_worked():
    g = _load("gat_hand.json")
    src = [e[0] for e in g["edges_src_to_dst"]]
    dst = [e[1] for e in g["edges_src_to_dst"]]
    rp, col, _ = _graph(g["n"], src, dst)
    ln3 = math.log(3.0)
    H = np.array([[ln3 if x == "ln3" else float(x) for x in row] for row in g["H"]])
    a_l = np.array(g["a_l"], dtype=np.float64)
    a_r = np.array(g["a_r"], dtype=np.float64)
    out = O.gat_layer(rp, col, H, np.eye(2), a_l, a_r, np.zeros(2), 1, "concat", "none",
                      g["neg_slope"])
    w0 = math.exp(-0.4) / (math.exp(-0.4) + 3.0)
    w1 = 3.0 / (math.exp(-0.4) + 3.0)
    want = np.array([[0.75 * ln3, 5.0], [-2.0, 1.0],
                     [w0 * -2.0 + w1 * ln3, w0 * 1.0 + w1 * 4.0], [0.0, 0.0]])
    np.testing.assert_allclose(out, want, rtol=1e-14, atol=1e-15)


def test_gat_head_mean_hand_worked():
    """Two heads averaged (the second GAT layer's merge), worked by hand in
    tests/golden/gat_mean_hand.json."""
    g = _load("gat_mean_hand.json")
    src = [e[0] for e in g["edges_src_to_dst"]]
    dst = [e[1] for e in g["edges_src_to_dst"]]
    rp, col, _ = _graph(g["n"], src, dst)
    ln3 = math.log(3.0)
    H = np.array([[ln3 if x == "ln3" else float(x) for x in row] for row in g["H"]])
    out = O.gat_layer(rp, col, H, np.eye(4), np.array(g["a_l"], dtype=np.float64),
                      np.array(g["a_r"], dtype=np.float64), np.array(g["b"], dtype=np.float64),
                      g["heads"], "mean", "none", g["neg_slope"])
    e = math.e
    w1, w2 = 1.0 / (1.0 + e), e / (1.0 + e)
    want = np.array([[(0.75 * ln3 + 6 * w1 + 10 * w2) / 2 + 0.5, (2.5 - 5 * w1) / 2 - 1.0],
                     [3.5, 4.0], [0.5, -1.0]])
    np.testing.assert_allclose(out, want, rtol=1e-14, atol=1e-15)


def test_gru_cell_equals_torch_grucell():
    """The GRU ApplyVertex (Fig. 2, GGNN) against torch.nn.GRUCell in float64
    with non-zero input and hidden weights and biases: gate order (r, z, n),
    the reset gate applied to h W_hn + b_hn, h' = (1 - z) n + z h."""
    import torch

    rng = np.random.default_rng(21)
    F, M = 5, 9
    a = rng.standard_normal((M, F))
    h = rng.standard_normal((M, F))
    W_ih = rng.standard_normal((F, 3 * F))
    W_hh = rng.standard_normal((F, 3 * F))
    b_ih = rng.standard_normal(3 * F)
    b_hh = rng.standard_normal(3 * F)
    cell = torch.nn.GRUCell(F, F, bias=True, dtype=torch.float64)
    with torch.no_grad():
        cell.weight_ih.copy_(torch.from_numpy(W_ih.T.copy()))
        cell.weight_hh.copy_(torch.from_numpy(W_hh.T.copy()))
        cell.bias_ih.copy_(torch.from_numpy(b_ih))
        cell.bias_hh.copy_(torch.from_numpy(b_hh))
        want = cell(torch.from_numpy(a), torch.from_numpy(h)).numpy()
    got = O.gru_cell(a, h, W_ih, b_ih, W_hh, b_hh)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------
# dense brute force on tiny graphs (multi-edges, self-loops, empty rows,
# star hub, chain)
# --------------------------------------------------------------------------
@pytest.mark.parametrize("case", tiny_graphs(), ids=lambda c: c[0])
def test_gather_sum_mean_equal_dense_product(case):
    name, n, src, dst = case
    rp, col, _ = _graph(n, src, dst)
    A = dense_adjacency(n, src, dst)
    rng = np.random.default_rng(1)
    S = rng.standard_normal((n, 7))
    np.testing.assert_allclose(O.gather(rp, col, S, "sum"), A @ S, rtol=1e-12, atol=1e-12)
    din = A.sum(axis=1)
    mean = np.where(din[:, None] > 0, (A @ S) / np.maximum(din, 1)[:, None], 0.0)
    np.testing.assert_allclose(O.gather(rp, col, S, "mean"), mean, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", tiny_graphs(), ids=lambda c: c[0])
def test_gather_max_equals_masked_max(case):
    name, n, src, dst = case
    rp, col, _ = _graph(n, src, dst)
    A = dense_adjacency(n, src, dst)
    rng = np.random.default_rng(2)
    S = rng.standard_normal((n, 5)).astype(np.float32)
    got = O.gather(rp, col, S, "max")
    for v in range(n):
        mask = A[v] > 0
        want = S[mask].max(axis=0) if mask.any() else np.zeros(5)
        assert np.array_equal(got[v], want.astype(np.float64))
        # invariant: a_v >= every neighbour's value, with equality attained
        if mask.any():
            assert np.all(got[v][None, :] >= S[mask])
            assert np.all(np.any(S[mask] == got[v][None, :], axis=0))


@pytest.mark.parametrize("case", tiny_graphs(), ids=lambda c: c[0])
def test_gcn_equals_dense_normalised_product(case):
    name, n, src, dst = case
    rp, col, _ = _graph(n, src, dst)
    A = dense_adjacency(n, src, dst)
    rng = np.random.default_rng(3)
    X = rng.standard_normal((n, 6))
    W = rng.standard_normal((6, 4))
    b = rng.standard_normal(4)
    din = A.sum(axis=1)
    dout = A.sum(axis=0)
    si = np.where(din > 0, 1.0 / np.sqrt(np.maximum(din, 1)), 0.0)
    so = np.where(dout > 0, 1.0 / np.sqrt(np.maximum(dout, 1)), 0.0)
    Ahat = si[:, None] * A * so[None, :]
    want = np.maximum(Ahat @ X @ W + b, 0.0)
    got = O.gcn_layer(rp, col, X, W, b, "relu")
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)
    got_tf = O.gcn_layer(rp, col, X, W, b, "relu", order="transform_first")
    np.testing.assert_allclose(got_tf, got, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", tiny_graphs(), ids=lambda c: c[0])
def test_attention_equals_dense_masked_softmax(case):
    name, n, src, dst = case
    rp, col, _ = _graph(n, src, dst)
    A = dense_adjacency(n, src, dst)
    K, D = 2, 3
    rng = np.random.default_rng(4)
    Z = rng.standard_normal((n, K * D))
    el = rng.standard_normal((n, K))
    er = rng.standard_normal((n, K))
    got, alphas = O.attention_gather(rp, col, Z, el, er, K, 0.2, return_alpha=True)
    for v in range(n):
        for k in range(K):
            s = el[:, k] + er[v, k]
            s = np.where(s > 0, s, 0.2 * s)
            w = A[v] * np.exp(s - s.max())        # multiplicity-weighted
            if A[v].sum() == 0:
                np.testing.assert_array_equal(got[v, k * D:(k + 1) * D], 0.0)
                continue
            alpha = w / w.sum()
            want = alpha @ Z[:, k * D:(k + 1) * D]
            np.testing.assert_allclose(got[v, k * D:(k + 1) * D], want, rtol=1e-12, atol=1e-12)
        # invariant: weights sum to 1 per destination and head
        if len(alphas[v]):
            d = len(alphas[v])
            assert np.all(np.abs(alphas[v].sum(axis=0) - 1.0) <= d * 2.0 ** -52 + 1e-15)


def test_gat_with_zero_attention_is_mean_aggregation():
    for name, n, src, dst in tiny_graphs():
        rp, col, _ = _graph(n, src, dst)
        rng = np.random.default_rng(5)
        K, D = 4, 2
        H = rng.standard_normal((n, 5))
        W = rng.standard_normal((5, K * D))
        zero = np.zeros((K, D))
        got = O.gat_layer(rp, col, H, W, zero, zero, np.zeros(K * D), K, "concat", "none")
        want = O.gather(rp, col, H @ W, "mean")
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", tiny_graphs(), ids=lambda c: c[0])
def test_gated_layer_equals_edge_loop(case):
    """Brute force straight from the edge list: each edge computes its gate
    from [h_u | h_v | e_uv] and adds gate * h_u into its destination."""
    name, n, src, dst = case
    rp, col, order = _graph(n, src, dst)
    F, Fe = 3, 2
    rng = np.random.default_rng(6)
    H = rng.standard_normal((n, F))
    E_list = rng.standard_normal((len(src), Fe))      # per edge-list entry
    E_csr = E_list[order]                             # CSR order
    W_e = rng.standard_normal((2 * F + Fe, F))
    b_e = rng.standard_normal(F)
    W_ih = rng.standard_normal((F, 3 * F))
    W_hh = rng.standard_normal((F, 3 * F))
    b_ih = rng.standard_normal(3 * F)
    b_hh = rng.standard_normal(3 * F)
    a = np.zeros((n, F))
    for e, (u, v) in enumerate(zip(src, dst)):
        x = np.concatenate([H[u], H[v], E_list[e]])
        gate = 1.0 / (1.0 + np.exp(-(x @ W_e + b_e)))
        a[v] += gate * H[u]
    got = O.gated_gru_layer(rp, col, H, E_csr, W_e, b_e, W_ih, b_ih, W_hh, b_hh)
    # textbook GRU cell, one vertex at a time
    want = np.zeros((n, F))
    for v in range(n):
        gi = a[v] @ W_ih + b_ih
        gh = H[v] @ W_hh + b_hh
        r = 1 / (1 + np.exp(-(gi[:F] + gh[:F])))
        z = 1 / (1 + np.exp(-(gi[F:2 * F] + gh[F:2 * F])))
        nn = np.tanh(gi[2 * F:] + r * gh[2 * F:])
        want[v] = (1 - z) * nn + z * H[v]
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", tiny_graphs(), ids=lambda c: c[0])
def test_sage_pool_equals_brute_force(case):
    name, n, src, dst = case
    rp, col, _ = _graph(n, src, dst)
    A = dense_adjacency(n, src, dst)
    rng = np.random.default_rng(8)
    F = 4
    X = rng.standard_normal((n, F))
    Wp = rng.standard_normal((F, F))
    bp = rng.standard_normal(F)
    W = rng.standard_normal((2 * F, 3))
    b = rng.standard_normal(3)
    P = np.maximum(X @ Wp + bp, 0)
    want = np.zeros((n, 3))
    for v in range(n):
        nb = np.flatnonzero(A[v] > 0)
        agg = P[nb].max(axis=0) if len(nb) else np.zeros(F)
        want[v] = np.concatenate([X[v], agg]) @ W + b
    got = O.sage_pool_layer(rp, col, X, Wp, bp, W, b)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------
# closed forms and special cases
# --------------------------------------------------------------------------
def test_closed_forms_of_sum_mean_and_gcn():
    for name, n, src, dst in tiny_graphs():
        rp, col, _ = _graph(n, src, dst)
        ones = np.ones((n, 3))
        din = np.bincount(dst, minlength=n).astype(np.float64)
        np.testing.assert_array_equal(O.gather(rp, col, ones, "sum")[:, 0], din)
        np.testing.assert_array_equal(O.gather(rp, col, ones, "mean")[:, 0],
                                      (din > 0).astype(np.float64))
    # d-regular graph with self-loops: circulant, every vertex has in- and
    # out-degree d; GCN-normalised aggregation of all-ones gives 1
    n, d = 30, 5
    src, dst = [], []
    for v in range(n):
        for j in range(d):
            src.append((v + j) % n)
            dst.append(v)
    rp, col, _ = _graph(n, src, dst)
    y = O.gcn_layer(rp, col, np.ones((n, 2)), np.eye(2), np.zeros(2), "none")
    np.testing.assert_allclose(y, 1.0, rtol=1e-15)


def test_gru_closed_forms():
    rng = np.random.default_rng(9)
    F = 4
    h = rng.standard_normal((6, F))
    a = rng.standard_normal((6, F))
    Z3 = np.zeros((F, 3 * F))
    # all weights and biases zero: r = z = 1/2, n = 0 -> h' = h / 2
    np.testing.assert_allclose(O.gru_cell(a, h, Z3, np.zeros(3 * F), Z3, np.zeros(3 * F)),
                               0.5 * h, rtol=1e-15)
    # large update-gate bias: z -> 1, h' -> h
    b = np.zeros(3 * F)
    b[F:2 * F] = 60.0
    np.testing.assert_allclose(O.gru_cell(a, h, Z3, b, Z3, np.zeros(3 * F)), h, atol=1e-12)
    # large negative update-gate bias and zero reset path: h' = tanh(a W_in)
    W_ih = rng.standard_normal((F, 3 * F))
    b = np.zeros(3 * F)
    b[F:2 * F] = -60.0
    got = O.gru_cell(a, h, W_ih, b, Z3, np.zeros(3 * F))
    np.testing.assert_allclose(got, np.tanh(a @ W_ih[:, 2 * F:]), atol=1e-12)


def test_zero_gate_weights_give_half_sum():
    for name, n, src, dst in tiny_graphs():
        rp, col, _ = _graph(n, src, dst)
        rng = np.random.default_rng(10)
        F = 3
        H = rng.standard_normal((n, F))
        E = rng.standard_normal((len(src), 2))
        W_e = np.zeros((2 * F + 2, F))
        I3 = np.zeros((F, 3 * F))
        I3[:, 2 * F:] = np.eye(F)
        # with W_ih = [0 | 0 | I], W_hh = 0, b_z = -60: h' = tanh(a)
        b = np.zeros(3 * F)
        b[F:2 * F] = -60.0
        got = O.gated_gru_layer(rp, col, H, E, W_e, np.zeros(F), I3, b,
                                np.zeros((F, 3 * F)), np.zeros(3 * F))
        a = 0.5 * O.gather(rp, col, H, "sum")
        np.testing.assert_allclose(got, np.tanh(a), atol=1e-12)


def test_dense_on_small_integers_is_exact():
    rng = np.random.default_rng(11)
    A = rng.integers(-8, 9, (9, 13))
    W = rng.integers(-8, 9, (13, 5))
    want = [[sum(int(A[i, k]) * int(W[k, j]) for k in range(13)) for j in range(5)]
            for i in range(9)]
    assert np.array_equal(O.dense(A, W), np.array(want, dtype=np.float64))


def test_activations_textbook():
    x = np.array([-3.0, -0.0, 0.0, 2.5])
    assert np.array_equal(O.relu(x), [0.0, 0.0, 0.0, 2.5])
    assert not np.any(np.signbit(O.relu(x)))   # no -0 reaches a max reduction
    np.testing.assert_allclose(O.elu(x), [math.exp(-3) - 1, 0, 0, 2.5], rtol=1e-15)
    np.testing.assert_allclose(O.leaky_relu(x, 0.2), [-0.6, 0, 0, 2.5], rtol=1e-15)
    np.testing.assert_allclose(O.sigmoid(np.array([0.0, math.log(3)])), [0.5, 0.75], rtol=1e-15)


# --------------------------------------------------------------------------
# permutation equivariance
# --------------------------------------------------------------------------
def _relabelled(n, src, dst, pi):
    return [int(pi[u]) for u in src], [int(pi[v]) for v in dst]


def test_permutation_equivariance_all_layers():
    name, n, src, dst = tiny_graphs()[3]
    rng = np.random.default_rng(12)
    pi = rng.permutation(n)                 # vertex x is renamed pi[x]
    inv = np.argsort(pi)
    rp, col, order = _graph(n, src, dst)
    s2, d2 = _relabelled(n, src, dst, pi)
    rp2, col2, order2 = _graph(n, s2, d2)
    X = rng.standard_normal((n, 6))
    X2 = X[inv]                             # row pi[x] of X2 is row x of X
    W = rng.standard_normal((6, 4))
    b = rng.standard_normal(4)
    y = O.gcn_layer(rp, col, X, W, b, "relu")
    y2 = O.gcn_layer(rp2, col2, X2, W, b, "relu")
    np.testing.assert_allclose(y2[pi], y, rtol=1e-12, atol=1e-12)
    # GAT
    K, D = 2, 2
    al = rng.standard_normal((K, D))
    ar = rng.standard_normal((K, D))
    Wg = rng.standard_normal((6, K * D))
    y = O.gat_layer(rp, col, X, Wg, al, ar, np.zeros(K * D), K, "concat", "elu")
    y2 = O.gat_layer(rp2, col2, X2, Wg, al, ar, np.zeros(K * D), K, "concat", "elu")
    np.testing.assert_allclose(y2[pi], y, rtol=1e-12, atol=1e-12)
    # SAGE max: exact
    Wp = rng.standard_normal((6, 6))
    bp = rng.standard_normal(6)
    Wc = rng.standard_normal((12, 3))
    y = O.sage_pool_layer(rp, col, X, Wp, bp, Wc, np.zeros(3))
    y2 = O.sage_pool_layer(rp2, col2, X2, Wp, bp, Wc, np.zeros(3))
    np.testing.assert_allclose(y2[pi], y, rtol=1e-12, atol=1e-12)
    # max gather itself is bit-exact under relabelling
    m = O.gather(rp, col, X, "max")
    m2 = O.gather(rp2, col2, X2, "max")
    assert np.array_equal(m2[pi], m)
    # gated: edge features follow their edges
    E_list = rng.standard_normal((len(src), 2))
    F = 6
    W_e = rng.standard_normal((2 * F + 2, F))
    args = (rng.standard_normal(F), rng.standard_normal((F, 3 * F)), rng.standard_normal(3 * F),
            rng.standard_normal((F, 3 * F)), rng.standard_normal(3 * F))
    y = O.gated_gru_layer(rp, col, X, E_list[order], W_e, *args)
    y2 = O.gated_gru_layer(rp2, col2, X2, E_list[order2], W_e, *args)
    np.testing.assert_allclose(y2[pi], y, rtol=1e-12, atol=1e-12)


# --------------------------------------------------------------------------
# two-layer compositions use the pinned layers (parity of the composition is
# otherwise unpinned); rows= restriction agrees with the full evaluation
# --------------------------------------------------------------------------
def test_row_restricted_evaluation_matches_full():
    from synth import configs as C

    g = C.build("gcn_er", small=True)
    full = O.gcn_2layer(g)
    rows = np.array([0, 5, 17, 1999, 1234])
    np.testing.assert_allclose(O.gcn_2layer(g, rows=rows), full[rows], rtol=1e-13, atol=1e-13)
    g = C.build("gat_ba", small=True, n=600)
    full = O.gat_2layer(g)
    rows = np.array([0, 3, 599, 250])
    np.testing.assert_allclose(O.gat_2layer(g, rows=rows), full[rows], rtol=1e-13, atol=1e-13)


# --------------------------------------------------------------------------
# layout: integer invariants and a hand-worked plan
# --------------------------------------------------------------------------
def test_layout_hand_worked():
    # rows: 0 has 5 edges, 1 has 0, 2 has 2, 3 has 5, 4 has 1
    rp = np.array([0, 5, 5, 7, 12, 13])
    col = np.array([1, 1, 2, 3, 4, 0, 0, 4, 4, 4, 4, 4, 2])
    p = O.plan(rp, col, 5, seg_len=2, block_cost=6, row_cost=1)
    assert p["d_in"].tolist() == [5, 0, 2, 5, 1]
    assert p["d_out"].tolist() == [2, 2, 2, 1, 6]
    assert p["perm"].tolist() == [0, 3, 2, 4, 1]          # degree desc, id asc
    # segments of <= 2 edges in perm order: row 0 -> [0,2) [2,4) [4,5);
    # row 3 -> [7,9) [9,11) [11,12); row 2 -> [5,7); row 4 -> [12,13); row 1 -> [5,5)
    assert p["seg_row"].tolist() == [0, 0, 0, 3, 3, 3, 2, 4, 1]
    assert p["seg_beg"].tolist() == [0, 2, 4, 7, 9, 11, 5, 12, 5]
    assert p["seg_end"].tolist() == [2, 4, 5, 9, 11, 12, 7, 13, 5]
    assert p["row_seg_first"].tolist() == [0, 3, 6, 7, 8, 9]
    # costs (edges + 1): 3 3 2 3 3 2 3 2 1; cost before each segment:
    # 0 3 6 8 11 14 16 19 21 -> //6: 0 0 1 1 1 2 2 3 3
    assert p["block_ptr"].tolist() == [0, 2, 5, 7, 9]
    assert p["n_split"] == 2


def test_layout_invariants_on_power_law_graph():
    from synth import configs as C

    g = C.build("sage_rmat", small=True)
    rp = g["row_ptr"].astype(np.int64)
    col = g["col_idx"]
    n = g["num_vertices"]
    E = g["num_edges"]
    T, B, c = 64, 1024, 4
    p = O.plan(rp, col, n, T, B, c)
    assert p["d_in"].sum() == E and p["d_out"].sum() == E
    assert np.array_equal(np.sort(p["perm"]), np.arange(n))
    key = sorted(range(n), key=lambda v: (-int(rp[v + 1] - rp[v]), v))
    assert p["perm"].tolist() == key
    # every CSR entry is covered exactly once by the segments
    cover = np.zeros(E, dtype=np.int64)
    for b_, e_ in zip(p["seg_beg"], p["seg_end"]):
        cover[b_:e_] += 1
        assert 0 <= e_ - b_ <= T
    assert np.all(cover == 1)
    for r, b_, e_ in zip(p["seg_row"], p["seg_beg"], p["seg_end"]):
        assert rp[r] <= b_ <= e_ <= rp[r + 1]
    # blocks tile the segment list and each one costs < block_cost + max cost
    bp = p["block_ptr"]
    assert bp[0] == 0 and bp[-1] == len(p["seg_row"]) and np.all(np.diff(bp) > 0)
    cost = p["seg_end"] - p["seg_beg"] + c
    for k in range(len(bp) - 1):
        assert cost[bp[k]:bp[k + 1]].sum() < B + cost.max()
    # split rows are exactly the rows with more than T in-edges, and come first
    assert p["n_split"] == int(np.sum(p["d_in"] > T))
    assert np.all(p["d_in"][p["perm"][:p["n_split"]]] > T)


# --------------------------------------------------------------------------
# planted mistakes: each plausible bug in the oracle breaks one of the pins
# --------------------------------------------------------------------------
def _pins_pass():
    try:
        test_gcn_hand_worked()
        test_gat_hand_worked()
        for case in tiny_graphs():
            test_gather_sum_mean_equal_dense_product(case)
            test_gcn_equals_dense_normalised_product(case)
            test_attention_equals_dense_masked_softmax(case)
            test_gated_layer_equals_edge_loop(case)
            test_sage_pool_equals_brute_force(case)
            test_gather_max_equals_masked_max(case)
        test_closed_forms_of_sum_mean_and_gcn()
        test_gru_closed_forms()
        test_gat_head_mean_hand_worked()
        test_gru_cell_equals_torch_grucell()
    except AssertionError:
        return False
    return True


def test_pins_pass_unmutated():
    assert _pins_pass()


def _gat_mean_over_dims(orig):
    """GAT head merge averaging each head's dims instead of the heads (same
    output shape when heads == head dims)."""
    def f(row_ptr, col_idx, H, W, a_l, a_r, b, heads, merge, act, neg_slope=0.2, rows=None):
        if merge != "mean":
            return orig(row_ptr, col_idx, H, W, a_l, a_r, b, heads, merge, act, neg_slope, rows)
        F = W.shape[1]
        o = orig(row_ptr, col_idx, H, W, a_l, a_r, np.zeros(F), heads, "concat", "none",
                 neg_slope, rows)
        return O.ACTS[act](o.reshape(-1, heads, F // heads).mean(axis=2)
                           + np.asarray(b, dtype=np.float64)[None, :])
    return f


def _gru_mutant(kind):
    """GRU cells with a misplaced reset gate or hidden bias."""
    def f(a, h, W_ih, b_ih, W_hh, b_hh):
        F = h.shape[1]
        gi = a @ W_ih + b_ih[None, :]
        gh_w = h @ W_hh
        gh = gh_w + b_hh[None, :]
        r = 1.0 / (1.0 + np.exp(-(gi[:, :F] + gh[:, :F])))
        z = 1.0 / (1.0 + np.exp(-(gi[:, F:2 * F] + gh[:, F:2 * F])))
        if kind == "reset_on_input":      # r gates the input side instead
            n = np.tanh(r * gi[:, 2 * F:] + gh[:, 2 * F:])
        else:                             # b_hn added outside the reset gate
            n = np.tanh(gi[:, 2 * F:] + r * gh_w[:, 2 * F:] + b_hh[None, 2 * F:])
        return (1.0 - z) * n + z * h
    return f


MUTANTS = {
    # GAT layer 2 averaging over each head's dims instead of over the heads
    "gat_mean_over_dims": lambda O_: setattr(O_, "gat_layer", _gat_mean_over_dims(O_.gat_layer)),
    # GRU reset gate applied to the input side
    "gru_reset_on_input": lambda O_: setattr(O_, "gru_cell", _gru_mutant("reset_on_input")),
    # GRU hidden bias b_hn outside the reset gate
    "gru_bhn_outside_reset": lambda O_: setattr(O_, "gru_cell", _gru_mutant("bhn_outside")),
    # dropped destination scaling in GCN
    "gcn_no_din": lambda O_: setattr(O_, "in_degrees", lambda rp: np.ones(len(rp) - 1, np.int64)),
    # wrong sign in LeakyReLU
    "leaky_sign": lambda O_: setattr(O_, "leaky_relu", lambda x, s: np.where(x > 0, x, -s * x)),
    # wrong sign inside the sigmoid (the gated edge MPNN's gate)
    "sigmoid_sign": lambda O_: setattr(O_, "sigmoid", lambda x: 1.0 / (1.0 + np.exp(x))),
    # transposed operand in the dense transform
    "dense_transpose": lambda O_: setattr(
        O_, "dense", (lambda orig: (lambda A, W, **k: orig(A, W.T if W.shape[0] == W.shape[1] else W, **k)))(O_.dense)),
    # degree scaling d^-1 instead of d^-1/2 (GCN normalisation)
    "degree_scale_sq": lambda O_: setattr(O_, "degree_scale", lambda d: np.where(np.asarray(d) > 0, 1.0 / np.maximum(np.asarray(d, float), 1), 0.0)),
}


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_planted_mistake_is_caught(mutant, monkeypatch):
    import oracle.saga_oracle as mod

    saved = {k: getattr(mod, k) for k in ("in_degrees", "leaky_relu", "sigmoid", "dense", "degree_scale",
                                           "gat_layer", "gru_cell")}
    try:
        MUTANTS[mutant](mod)
        assert not _pins_pass(), f"mutant {mutant} survived the pins"
    finally:
        for k, v in saved.items():
            setattr(mod, k, v)


def test_rel_err_metric():
    r = np.array([1.0, -2.0, 0.0, 1e-9])
    y = r + np.array([1e-5, 0, 1e-6, 0])
    rms = math.sqrt((1 + 4 + 1e-18) / 4)
    # element 0: |r| = 1 < rms, so the floor applies; element 1 is exact
    assert abs(rel_err(y, r) - max(1e-5 / rms, 1e-6 / rms)) < 1e-15
