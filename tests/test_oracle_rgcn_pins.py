"""Pins of the oracle's R-GCN layer and typed layout (Table I, R-GCN row;
Sec. 3.2 "ApplyEdge": edges carry a type and the edges of one type share one
transform).  The layer is pinned to a hand-worked example, to a dense
per-relation adjacency product, to a closed form (the number of distinct
relation types entering a vertex), to the single-relation case (a mean
Gather followed by a linear map), and to invariance under relabelling of the
vertices and of the relation ids; planted mistakes each break one of them.
The typed layout (the library's own definition) is pinned to a hand-worked
example and to invariants.  CPU only."""
import json
import os

import numpy as np
import pytest

from helpers import dense_adjacency, edges_to_csr, tiny_graphs
from oracle import saga_oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _typed(n, src, dst, types):
    """CSR of an edge list plus its types in CSR order."""
    rp, col, order = edges_to_csr(n, src, dst)
    et = np.array([types[e] for e in order], dtype=np.int32)
    return rp, col, et


def _typed_tiny(R=3, seed=11):
    out = []
    rng = np.random.default_rng(seed)
    for name, n, src, dst in tiny_graphs():
        types = rng.integers(0, R, len(src)).tolist()
        out.append((name, n, src, dst, types))
    return out


def _weights(R, Fi, Fo, seed):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((R, Fi, Fo)), rng.standard_normal((Fi, Fo)),
            rng.standard_normal(Fo))


def test_rgcn_hand_worked():
    with open(os.path.join(GOLDEN, "rgcn_hand.json")) as f:
        g = json.load(f)
    src, dst, ty = zip(*g["edges_src_dst_type"])
    rp, col, et = _typed(g["n"], list(src), list(dst), list(ty))
    lay = g["layout"]
    assert rp.tolist() == lay["csr_row_ptr"] and col.tolist() == lay["csr_col_idx"]
    assert et.tolist() == lay["csr_etype"]
    X, Wr, Ws, b = (np.array(g[k], dtype=np.float64) for k in ("X", "W_rel", "W_self", "b"))
    pre = O.rgcn_layer(rp, col, et, X, Wr, Ws, b)
    assert np.array_equal(pre, np.array(g["pre_activation"]))
    out = O.rgcn_layer(rp, col, et, X, Wr, Ws, b, act="relu")
    assert np.array_equal(out, np.array(g["relu_output"]))


@pytest.mark.parametrize("case", _typed_tiny(), ids=lambda c: c[0])
def test_rgcn_equals_dense_relational_product(case):
    """Y = X W_self + b + sum_r C_r^-1 A_r X W_r with A_r the dense
    adjacency of the type-r edges (multiplicities) and C_r its row sums
    (rows with C_r = 0 contribute nothing)."""
    name, n, src, dst, types = case
    R, Fi, Fo = 3, 5, 4
    rp, col, et = _typed(n, src, dst, types)
    X = np.random.default_rng(3).standard_normal((n, Fi))
    Wr, Ws, b = _weights(R, Fi, Fo, 4)
    want = X @ Ws + b[None, :]
    for r in range(R):
        sel = [e for e in range(len(src)) if types[e] == r]
        A = dense_adjacency(n, [src[e] for e in sel], [dst[e] for e in sel])
        c = A.sum(axis=1)
        inv = np.where(c > 0, 1.0 / np.maximum(c, 1), 0.0)
        want = want + (inv[:, None] * (A @ X)) @ Wr[r]
    got = O.rgcn_layer(rp, col, et, X, Wr, Ws, b)
    assert np.allclose(got, want, rtol=0, atol=1e-12 * max(1.0, np.abs(want).max()))


def test_rgcn_counts_distinct_relations():
    """x = 1 (one column), W_r = 1 for every r, W_self = 0, b = 0: each
    relation present among v's in-edges contributes exactly 1, so y_v is the
    number of distinct types entering v."""
    for name, n, src, dst, types in _typed_tiny(R=4, seed=5):
        rp, col, et = _typed(n, src, dst, types)
        y = O.rgcn_layer(rp, col, et, np.ones((n, 1)), np.ones((4, 1, 1)), np.zeros((1, 1)),
                         np.zeros(1))
        want = [len({types[e] for e in range(len(src)) if dst[e] == v}) for v in range(n)]
        assert np.array_equal(y[:, 0], np.array(want, dtype=np.float64)), name


@pytest.mark.parametrize("case", _typed_tiny(R=1), ids=lambda c: c[0])
def test_single_relation_is_mean_gather_then_linear(case):
    name, n, src, dst, types = case
    rp, col, et = _typed(n, src, dst, types)
    X = np.random.default_rng(8).standard_normal((n, 6))
    Wr, Ws, b = _weights(1, 6, 3, 9)
    want = O.dense(X, Ws, bias=b) + O.dense(O.gather(rp, col, X, "mean"), Wr[0])
    got = O.rgcn_layer(rp, col, et, X, Wr, Ws, b)
    assert np.allclose(got, want, rtol=0, atol=1e-12)


def test_rgcn_relabelling_invariances():
    from synth import configs as C

    g = C.build("rgcn_rmat", small=True)
    n, R = g["num_vertices"], g["num_rel"]
    rows = np.arange(0, n, 7)
    base = O.rgcn_layer_of(g, rows=rows)
    # relation ids permuted together with their weights: same output
    pr = np.random.default_rng(2).permutation(R)
    g2 = dict(g)
    g2["etype"] = pr[g["etype"]].astype(np.int32)
    W2 = np.empty_like(g["W_rel"])
    W2[pr] = g["W_rel"]
    g2["W_rel"] = W2
    assert np.allclose(O.rgcn_layer_of(g2, rows=rows), base, rtol=0, atol=1e-11)
    # vertices relabelled by pi: output rows move with them
    pi = np.random.default_rng(3).permutation(n)
    rp, col = g["row_ptr"].astype(np.int64), g["col_idx"]
    dst = np.repeat(np.arange(n), np.diff(rp))
    src2, dst2 = pi[col], pi[dst]
    order = np.lexsort((np.arange(len(col)), src2, dst2))
    rp2 = np.zeros(n + 1, np.int64)
    np.cumsum(np.bincount(dst2, minlength=n), out=rp2[1:])
    X2 = np.empty_like(g["X"])
    X2[pi] = g["X"]
    y2 = O.rgcn_layer(rp2, src2[order], g["etype"][order], X2, g["W_rel"], g["W_self"], g["b"],
                      act="relu", rows=pi[rows])
    assert np.allclose(y2, base, rtol=0, atol=1e-11)


def test_rel_layout_hand_worked():
    with open(os.path.join(GOLDEN, "rgcn_hand.json")) as f:
        g = json.load(f)
    lay = g["layout"]
    L = O.rel_layout(lay["csr_row_ptr"], lay["csr_col_idx"], lay["csr_etype"], g["num_rel"],
                     g["layout_tile"])
    for k in ("rel_count", "rel_ptr", "pair_src", "edge_pair"):
        assert L[k].tolist() == lay[k], k
    assert L["edge_norm"].tolist() == lay["edge_norm"]


def test_rel_layout_invariants():
    from synth import configs as C

    g = C.build("rgcn_rmat", small=True)
    R, tile = g["num_rel"], 128
    rp, col, et = g["row_ptr"].astype(np.int64), g["col_idx"].astype(np.int64), g["etype"]
    L = O.rel_layout(rp, col, et, R, tile)
    rel_ptr, ps = L["rel_ptr"], L["pair_src"]
    assert np.all(rel_ptr % tile == 0) and np.all(np.diff(rel_ptr) >= L["rel_count"])
    assert np.all(np.diff(rel_ptr) < L["rel_count"] + tile)
    for r in range(R):
        q = ps[rel_ptr[r]:rel_ptr[r + 1]]
        real, pad = q[:L["rel_count"][r]], q[L["rel_count"][r]:]
        assert np.all(np.diff(real) > 0) and np.all(pad == -1)
    # every edge points at its own (relation, source) pair; the pairs are
    # exactly the distinct (relation, source) combinations of the edges
    ep = L["edge_pair"]
    assert np.array_equal(ps[ep], col)
    assert np.all(ep >= rel_ptr[et]) and np.all(ep < rel_ptr[et] + L["rel_count"][et])
    assert L["rel_count"].sum() == len({(int(a), int(b)) for a, b in zip(et, col)})
    # norms: 1 / (number of in-edges of the same row and type)
    dst = np.repeat(np.arange(len(rp) - 1), np.diff(rp))
    key = dst * R + et
    _, inv, cnt = np.unique(key, return_inverse=True, return_counts=True)
    assert np.array_equal(L["edge_norm"], (1.0 / cnt[inv]).astype(np.float32))


# --------------------------------------------------------------------------
# planted mistakes: each plausible bug in the oracle breaks one of the pins
# --------------------------------------------------------------------------
def _pins_pass():
    try:
        test_rgcn_hand_worked()
        for case in _typed_tiny():
            test_rgcn_equals_dense_relational_product(case)
        test_rgcn_counts_distinct_relations()
        for case in _typed_tiny(R=1):
            test_single_relation_is_mean_gather_then_linear(case)
    except AssertionError:
        return False
    return True


def test_pins_pass_unmutated():
    assert _pins_pass()


def _norm_by_in_degree(orig):
    # normalise by the whole in-degree instead of the per-relation count
    def f(row_ptr, etype, num_rel, rows=None):
        c = orig(row_ptr, etype, num_rel, rows=rows)
        return np.repeat(c.sum(axis=1, keepdims=True), num_rel, axis=1)
    return f


def _shift_relation(orig):
    # messages credited to the next relation's weight
    def f(*a, **k):
        return np.roll(orig(*a, **k), 1, axis=1)
    return f


def _no_norm(orig):
    def f(row_ptr, etype, num_rel, rows=None):
        return np.minimum(orig(row_ptr, etype, num_rel, rows=rows), 1)
    return f


def _transposed_dense(orig):
    def f(A, W, **k):
        W = np.asarray(W)
        return orig(A, W.T if W.shape[0] == W.shape[1] else W, **k)
    return f


MUTANTS = {
    "norm_by_in_degree": ("relation_counts", _norm_by_in_degree),
    "relation_shift": ("rel_gather", _shift_relation),
    "no_norm": ("relation_counts", _no_norm),
    "dense_transpose": ("dense", _transposed_dense),
}


@pytest.mark.parametrize("mutant", sorted(MUTANTS))
def test_planted_mistake_is_caught(mutant, monkeypatch):
    import oracle.saga_oracle as mod

    name, wrap = MUTANTS[mutant]
    monkeypatch.setattr(mod, name, wrap(getattr(mod, name)))
    assert not _pins_pass(), f"mutant {mutant} survived the pins"
