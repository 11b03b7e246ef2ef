"""CPU oracle for the SAGA-NN message-passing layer.  TEST INFRASTRUCTURE.

This module is the reference the GPU library is checked against.  Only the
test suite, the package smoke check and the benchmark's CPU-baseline leg may
import it; the library itself never does, and it shares no code with the HIP
path (it reads the same seeded inputs from ``synth`` and nothing else).

Everything is plain numpy in float64, written to be read against the paper:

* A GNN layer maps (adjacency, vertex embeddings, edge embeddings) to new
  embeddings (Sec. 2, "Model Survey").  It is decomposed into Scatter ->
  ApplyEdge -> Gather -> ApplyVertex (Sec. 2, "Model Decomposition", and the
  GGNN walk-through of Fig. 2).
* Per-model stage contents follow Table I (GCN, GAT, GGNN rows; the
  GraphSAGE row with a max-pool reduction, one of the simple reductions
  listed under "Survey Result").
* A fused sum-Gather equals the product of the edge-to-vertex adjacency and
  the edge-embedding matrix (Sec. 3.2, Gather paragraph, Fig. 7b).  The
  adjacency is held as a destination-major CSR: row v lists the sources of
  v's in-edges; multi-edges appear once per copy.

The graph-layout functions (degrees, degree order, segments, row blocks)
restate the layout rules of the library's plan (a scheduling structure the
paper motivates with the power-law degree skew and the degree-traversal
discussion of Sec. 3.2 / Fig. 8); their outputs are integers and are compared
bit for bit.

Readings where the paper is silent (each one is also listed in the design
notes of the repository):
  R1 GCN normalisation on directed graphs: message weight
     d_out(u)^-1/2 * d_in(v)^-1/2, degrees counted on the stored edges
     (self-loops included when the workload adds them).
  R2 empty in-neighbourhood: sum, mean, max and attention aggregates are 0.
  R3 association order of GCN: aggregate first, then transform (Table I
     order); ``order="transform_first"`` exists only as a self-check.
  R4 GAT: z = h W (no bias inside), el/er per head, LeakyReLU(0.2) score,
     softmax over the in-edges of each destination; layer 1 concatenates
     heads (+ bias, ELU), layer 2 averages heads (+ bias, no activation).
  R5 gated edge MPNN: gate = sigmoid([h_u | h_v | e_uv] W_e + b_e) per
     feature, message = gate * h_u, sum over in-edges; GRU update with gate
     order (r, z, n).
  R6 SAGE-pool: p_u = ReLU(h_u W_pool + b_pool), elementwise max over
     in-edges, y = [h_v | a_v] W + b, no activation.
  R7 ReLU(x) = x if x > 0 else +0.
  R8 GraphSAGE with the LSTM reduction (Table I, GraphSAGE row; Sec. 3.2
     "Gather"): the in-edges of v, in CSR order, are the input sequence of
     an LSTM that starts from h = c = 0; a_v is its final hidden state (0
     for an empty row).  Gate blocks in the order (i, f, g, o) of width H:
     [i|f|g|o] = x_t W_ih + b_ih + h W_hh + b_hh, c = f*c + i*g,
     h = o*tanh(c), with i, f, o sigmoids and g a tanh.  Then
     y_v = [x_v | a_v] W + b, no activation.
  R9 R-GCN (Table I, R-GCN row: Scatter takes the edge and its source,
     ApplyEdge is a per-edge MLP, Gather sums the in-edges and adds the
     vertex itself, ApplyVertex is a sum; Sec. 3.2 "ApplyEdge": every edge
     carries a type, and the edges of one type share one transform).  Each
     relation r has a weight W_r; the message of an in-edge u -> v of type r
     is x_u W_r / c(v, r), where c(v, r) counts the in-edges of v of type r
     (the per-relation mean of the relational GCN); the vertex's own term is
     x_v W_self; y_v = act(b + x_v W_self + sum of the messages).  The edge
     types are an int32 array aligned with the CSR entries.
"""
from __future__ import annotations

import numpy as np

# ==========================================================================
# Graph layout (integers, bit-exact)
# ==========================================================================


def in_degrees(row_ptr):
    """d_in(v): number of in-edges of v = length of CSR row v."""
    rp = np.asarray(row_ptr, dtype=np.int64)
    return (rp[1:] - rp[:-1]).astype(np.int64)


def out_degrees(col_idx, num_src):
    """d_out(u): number of CSR entries naming u as source."""
    d = np.zeros(num_src, dtype=np.int64)
    np.add.at(d, np.asarray(col_idx, dtype=np.int64), 1)
    return d


def degree_order(d_in):
    """Row order by in-degree, largest first; equal degrees by vertex id."""
    d = np.asarray(d_in, dtype=np.int64)
    ids = np.arange(d.shape[0], dtype=np.int64)
    return np.lexsort((ids, -d)).astype(np.int64)


def segments(row_ptr, perm, seg_len):
    """Cut each row (taken in ``perm`` order) into segments of at most
    ``seg_len`` edges; a row with d_in <= seg_len (including an empty row)
    is one segment.

    Returns (seg_row, seg_beg, seg_end, row_seg_first), where segment s
    covers CSR entries [seg_beg[s], seg_end[s]) of row seg_row[s] and the
    segments of perm position i are row_seg_first[i] .. row_seg_first[i+1]-1.
    """
    rp = np.asarray(row_ptr, dtype=np.int64)
    perm = np.asarray(perm, dtype=np.int64)
    d = rp[perm + 1] - rp[perm]
    nseg = np.maximum(1, (d + seg_len - 1) // seg_len)
    first = np.zeros(perm.shape[0] + 1, dtype=np.int64)
    np.cumsum(nseg, out=first[1:])
    seg_row = np.repeat(perm, nseg)
    j = np.arange(first[-1], dtype=np.int64) - np.repeat(first[:-1], nseg)
    seg_beg = rp[seg_row] + j * seg_len
    seg_end = np.minimum(seg_beg + seg_len, rp[seg_row + 1])
    return seg_row, seg_beg, seg_end, first


def row_blocks(seg_beg, seg_end, block_cost, row_cost):
    """Partition the segment list into blocks of consecutive segments.

    Segment s costs (edges + row_cost).  With P(s) the total cost of the
    segments before s, segment s opens a new block when s = 0 or
    floor(P(s)/block_cost) differs from floor(P(s-1)/block_cost).
    Returns block_ptr: block b holds segments block_ptr[b] .. block_ptr[b+1]-1.
    """
    cost = (np.asarray(seg_end, np.int64) - np.asarray(seg_beg, np.int64)) + row_cost
    S = cost.shape[0]
    before = np.zeros(S, dtype=np.int64)
    if S > 1:
        np.cumsum(cost[:-1], out=before[1:])
    bid = before // block_cost
    opens = np.ones(S, dtype=bool)
    opens[1:] = bid[1:] != bid[:-1]
    return np.concatenate([np.flatnonzero(opens), [S]]).astype(np.int64)


def plan(row_ptr, col_idx, num_src, seg_len, block_cost, row_cost):
    """All layout arrays at once (dict of int64 arrays)."""
    d_in = in_degrees(row_ptr)
    d_out = out_degrees(col_idx, num_src)
    perm = degree_order(d_in)
    seg_row, seg_beg, seg_end, first = segments(row_ptr, perm, seg_len)
    blocks = row_blocks(seg_beg, seg_end, block_cost, row_cost)
    n_split = int(np.count_nonzero((first[1:] - first[:-1]) > 1))
    return dict(d_in=d_in, d_out=d_out, perm=perm, seg_row=seg_row,
                seg_beg=seg_beg, seg_end=seg_end, row_seg_first=first,
                block_ptr=blocks, n_split=n_split)


# ==========================================================================
# Elementwise functions
# ==========================================================================


def relu(x):
    return np.where(x > 0, x, 0.0)


def elu(x):
    return np.where(x > 0, x, np.expm1(np.minimum(x, 0.0)))


def leaky_relu(x, slope):
    return np.where(x > 0, x, slope * x)


def sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


ACTS = {
    "none": lambda x: x,
    "relu": relu,
    "elu": elu,
    "sigmoid": sigmoid,
    "tanh": np.tanh,
}


def _f64(a):
    return np.asarray(a, dtype=np.float64)


def _rows_arg(rows, n):
    return np.arange(n, dtype=np.int64) if rows is None else np.asarray(rows, dtype=np.int64)


# ==========================================================================
# ApplyVertex: dense per-vertex transform (Sec. 3.2 ApplyVertex; Table III)
# ==========================================================================


def dense(A, W, bias=None, act="none", row_scale=None):
    """act(row_scale * (A W) + bias), all in float64."""
    Y = _f64(A) @ _f64(W)
    if row_scale is not None:
        Y = Y * _f64(row_scale)[:, None]
    if bias is not None:
        Y = Y + _f64(bias)[None, :]
    return ACTS[act](Y)


def degree_scale(deg):
    """deg^-1/2, and 0 where deg = 0."""
    deg = _f64(deg)
    out = np.zeros_like(deg)
    nz = deg > 0
    out[nz] = 1.0 / np.sqrt(deg[nz])
    return out


# ==========================================================================
# Scatter + ApplyEdge + Gather primitives (Sec. 3.2; Table I Gather column)
# ==========================================================================


def gather(row_ptr, col_idx, S, reduce, rows=None, src_scale=None):
    """Per destination v: reduce the messages of its in-edges.

    The message of edge (u -> v) is row u of S, times src_scale[u] if given.
    reduce: "sum", "mean" (sum / d_in), "max" (elementwise).  An empty row
    gives 0 (R2).  Returns len(rows) x F float64.
    """
    rp = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col_idx, dtype=np.int64)
    rows = _rows_arg(rows, rp.shape[0] - 1)
    S = np.asarray(S)
    out = np.zeros((rows.shape[0], S.shape[1]), dtype=np.float64)
    for i, v in enumerate(rows):
        nb = col[rp[v]:rp[v + 1]]
        if nb.shape[0] == 0:
            continue
        msg = _f64(S[nb])
        if src_scale is not None:
            msg = msg * _f64(src_scale)[nb][:, None]
        if reduce == "sum":
            out[i] = msg.sum(axis=0)
        elif reduce == "mean":
            out[i] = msg.sum(axis=0) / nb.shape[0]
        elif reduce == "max":
            out[i] = msg.max(axis=0)
        else:
            raise ValueError(reduce)
    return out


def attention_gather(row_ptr, col_idx, Z, el, er, heads, neg_slope, rows=None,
                     return_alpha=False):
    """Edge-softmax attention Gather (Table I, GAT row).

    For each destination v and head k: score of edge (u -> v) is
    LeakyReLU(el[u,k] + er[v,k]); weights are the softmax of the scores over
    v's in-edges; the head-k output is the weighted sum of the sources'
    head-k slices of Z.  Empty row -> 0.  Returns len(rows) x (heads*D).
    """
    rp = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col_idx, dtype=np.int64)
    rows = _rows_arg(rows, rp.shape[0] - 1)
    F = Z.shape[1]
    D = F // heads
    out = np.zeros((rows.shape[0], F), dtype=np.float64)
    alphas = []
    for i, v in enumerate(rows):
        nb = col[rp[v]:rp[v + 1]]
        if nb.shape[0] == 0:
            alphas.append(np.zeros((0, heads)))
            continue
        s = leaky_relu(_f64(el[nb]) + _f64(er[v])[None, :], neg_slope)  # d x K
        m = s.max(axis=0)
        w = np.exp(s - m[None, :])
        alpha = w / w.sum(axis=0)[None, :]
        alphas.append(alpha)
        zn = _f64(Z[nb]).reshape(nb.shape[0], heads, D)
        out[i] = np.einsum("ek,ekd->kd", alpha, zn).reshape(F)
    if return_alpha:
        return out, alphas
    return out


# ==========================================================================
# Layers (Table I rows)
# ==========================================================================


def gcn_layer(row_ptr, col_idx, X, W, b, act, rows=None, order="aggregate_first"):
    """GCN layer (Table I: Gather = sum over in-edges, ApplyVertex = MLP).

    y_v = act(b + d_in(v)^-1/2 * sum_{u in N(v)} d_out(u)^-1/2 x_u W)   (R1)
    """
    n_dst = len(row_ptr) - 1
    d_in = in_degrees(row_ptr)
    d_out = out_degrees(col_idx, X.shape[0])
    rows = _rows_arg(rows, n_dst)
    if order == "aggregate_first":
        agg = gather(row_ptr, col_idx, X, "sum", rows=rows, src_scale=degree_scale(d_out))
        agg = agg * degree_scale(d_in)[rows][:, None]
        return dense(agg, W, bias=b, act=act)
    if order == "transform_first":
        Z = dense(X, W, row_scale=degree_scale(d_out))
        agg = gather(row_ptr, col_idx, Z, "sum", rows=rows)
        agg = agg * degree_scale(d_in)[rows][:, None]
        return ACTS[act](agg + _f64(b)[None, :])
    raise ValueError(order)


def gcn_2layer(g, X=None, W1=None, W2=None, rows=None):
    """Two GCN layers: ReLU after the first, raw output after the second.
    ``rows`` restricts the second layer's output rows (the first layer is
    evaluated on those rows' in-neighbours only)."""
    rp, col = g["row_ptr"], g["col_idx"]
    X = g["X"] if X is None else X
    W1 = g["W1"] if W1 is None else W1
    W2 = g["W2"] if W2 is None else W2
    n = len(rp) - 1
    if rows is None:
        H1 = gcn_layer(rp, col, X, W1, g["b1"], "relu")
        return gcn_layer(rp, col, H1, W2, g["b2"], "none")
    rows = np.asarray(rows, dtype=np.int64)
    rp64 = np.asarray(rp, dtype=np.int64)
    need = np.unique(np.concatenate([col[rp64[v]:rp64[v + 1]] for v in rows] + [rows]))
    H1 = np.zeros((n, W1.shape[1]), dtype=np.float64)
    H1[need] = gcn_layer(rp, col, X, W1, g["b1"], "relu", rows=need)
    return gcn_layer(rp, col, H1, W2, g["b2"], "none", rows=rows)


def gat_layer(row_ptr, col_idx, H, W, a_l, a_r, b, heads, merge, act,
              neg_slope=0.2, rows=None):
    """GAT layer (Table I: Scatter src & dst, ApplyEdge = attention score,
    Gather = attention over in-edges, ApplyVertex; reading R4).

    merge = "concat": act(concat_k o_k + b);  merge = "mean": mean_k o_k + b.
    """
    rp = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col_idx, dtype=np.int64)
    n_dst = rp.shape[0] - 1
    rows = _rows_arg(rows, n_dst)
    F = W.shape[1]
    D = F // heads
    need = np.unique(np.concatenate([col[rp[v]:rp[v + 1]] for v in rows] + [rows]))
    Z = np.zeros((H.shape[0], F), dtype=np.float64)
    Z[need] = dense(H[need], W)
    Zh = Z.reshape(-1, heads, D)
    el = np.einsum("nkd,kd->nk", Zh, _f64(a_l))
    er = np.einsum("nkd,kd->nk", Zh, _f64(a_r))
    o = attention_gather(rp, col, Z, el, er, heads, neg_slope, rows=rows)
    if merge == "concat":
        return ACTS[act](o + _f64(b)[None, :])
    if merge == "mean":
        return ACTS[act](o.reshape(-1, heads, D).mean(axis=1) + _f64(b)[None, :])
    raise ValueError(merge)


def gat_2layer(g, rows=None):
    """Layer 1: concat heads + ELU; layer 2: mean over heads, no activation."""
    rp, col = g["row_ptr"], g["col_idx"]
    K = g["heads"]
    n = len(rp) - 1
    if rows is None:
        H1 = gat_layer(rp, col, g["X"], g["W1"], g["al1"], g["ar1"], g["b1"], K,
                       "concat", "elu", g["neg_slope"])
        return gat_layer(rp, col, H1, g["W2"], g["al2"], g["ar2"], g["b2"], K,
                         "mean", "none", g["neg_slope"])
    rows = np.asarray(rows, dtype=np.int64)
    rp64 = np.asarray(rp, dtype=np.int64)
    col64 = np.asarray(col, dtype=np.int64)
    need = np.unique(np.concatenate([col64[rp64[v]:rp64[v + 1]] for v in rows] + [rows]))
    H1 = np.zeros((n, g["W1"].shape[1]), dtype=np.float64)
    H1[need] = gat_layer(rp, col, g["X"], g["W1"], g["al1"], g["ar1"], g["b1"], K,
                         "concat", "elu", g["neg_slope"], rows=need)
    return gat_layer(rp, col, H1, g["W2"], g["al2"], g["ar2"], g["b2"], K,
                     "mean", "none", g["neg_slope"], rows=rows)


def sage_pool_layer(row_ptr, col_idx, X, W_pool, b_pool, W, b, rows=None):
    """GraphSAGE layer with max-pool reduction (reading R6).

    p_u = ReLU(x_u W_pool + b_pool); a_v = elementwise max over in-edges of
    p_u (0 if none); y_v = [x_v | a_v] W + b.
    """
    rp = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col_idx, dtype=np.int64)
    rows = _rows_arg(rows, rp.shape[0] - 1)
    need = np.unique(np.concatenate([col[rp[v]:rp[v + 1]] for v in rows] + [np.zeros(0, np.int64)]))
    P = np.zeros((X.shape[0], W_pool.shape[1]), dtype=np.float64)
    if need.shape[0]:
        P[need] = dense(X[need], W_pool, bias=b_pool, act="relu")
    A = gather(rp, col, P, "max", rows=rows)
    cat = np.concatenate([_f64(X[rows]), A], axis=1)
    return dense(cat, W, bias=b)


def gated_gather(row_ptr, col_idx, H, E_feat, W_e, b_e, rows=None):
    """Scatter + ApplyEdge + Gather of the gated edge MPNN (the GGNN example
    of Fig. 2 and Table I, GGNN row; reading R5).

    Scatter: edge (u -> v) carries [h_u | h_v | e_uv];
    ApplyEdge: g = sigmoid([h_u | h_v | e_uv] W_e + b_e), m = g * h_u;
    Gather: a_v = sum of m over v's in-edges (0 if none).
    E_feat row e belongs to CSR entry e.
    """
    rp = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col_idx, dtype=np.int64)
    rows = _rows_arg(rows, rp.shape[0] - 1)
    F = H.shape[1]
    A = np.zeros((rows.shape[0], F), dtype=np.float64)
    for i, v in enumerate(rows):
        lo, hi = rp[v], rp[v + 1]
        if hi == lo:
            continue
        nb = col[lo:hi]
        hu = _f64(H[nb])
        hv = np.repeat(_f64(H[v])[None, :], hi - lo, axis=0)
        cat = np.concatenate([hu, hv, _f64(E_feat[lo:hi])], axis=1)
        gate = sigmoid(cat @ _f64(W_e) + _f64(b_e)[None, :])
        A[i] = (gate * hu).sum(axis=0)
    return A


def gated_gru_layer(row_ptr, col_idx, H, E_feat, W_e, b_e, W_ih, b_ih, W_hh,
                    b_hh, rows=None):
    """Gated edge MPNN layer: gated_gather, then the GRU ApplyVertex with
    input a_v and hidden state h_v (Fig. 2: GGNN's ApplyVertex is a GRU)."""
    rows = _rows_arg(rows, len(row_ptr) - 1)
    A = gated_gather(row_ptr, col_idx, H, E_feat, W_e, b_e, rows=rows)
    return gru_cell(A, _f64(H[rows]), W_ih, b_ih, W_hh, b_hh)


def gru_cell(a, h, W_ih, b_ih, W_hh, b_hh):
    """GRU update with input a and hidden h; column blocks (r, z, n):
    r = s(a W_ir + b_ir + h W_hr + b_hr), z = s(a W_iz + b_iz + h W_hz + b_hz),
    n = tanh(a W_in + b_in + r * (h W_hn + b_hn)), h' = (1 - z) n + z h."""
    F = h.shape[1]
    gi = _f64(a) @ _f64(W_ih) + _f64(b_ih)[None, :]
    gh = _f64(h) @ _f64(W_hh) + _f64(b_hh)[None, :]
    r = sigmoid(gi[:, :F] + gh[:, :F])
    z = sigmoid(gi[:, F:2 * F] + gh[:, F:2 * F])
    n = np.tanh(gi[:, 2 * F:] + r * gh[:, 2 * F:])
    return (1.0 - z) * n + z * _f64(h)


def gated_layer_of(g, rows=None):
    return gated_gru_layer(g["row_ptr"], g["col_idx"], g["H"], g["E_feat"], g["W_e"],
                           g["b_e"], g["W_ih"], g["b_ih"], g["W_hh"], g["b_hh"], rows=rows)


def sage_layer_of(g, rows=None):
    return sage_pool_layer(g["row_ptr"], g["col_idx"], g["X"], g["W_pool"], g["b_pool"],
                           g["W"], g["b"], rows=rows)


def lstm_gather(row_ptr, col_idx, X, W_ih, b_ih, W_hh, b_hh, rows=None):
    """LSTM reduction over each destination's in-edges (reading R8).

    The paper names this Gather as the one that cannot be fused: it treats
    the in-edges of a vertex as a sequence (Sec. 3.2, Gather paragraph).
    For row v with sources u_1 .. u_d in CSR order, starting from h = c = 0:
        [i | f | g | o] = x_{u_t} W_ih + b_ih + h W_hh + b_hh
        i, f, o = sigmoid(.), g = tanh(.)
        c = f * c + i * g;  h = o * tanh(c)
    and a_v = h after the last step (0 for an empty row).
    """
    rp = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col_idx, dtype=np.int64)
    rows = _rows_arg(rows, rp.shape[0] - 1)
    Wi, Wh = _f64(W_ih), _f64(W_hh)
    b = _f64(b_ih) + _f64(b_hh)
    H = Wh.shape[0]
    A = np.zeros((rows.shape[0], H), dtype=np.float64)
    for n, v in enumerate(rows):
        nb = col[rp[v]:rp[v + 1]]
        if nb.shape[0] == 0:
            continue
        # input contributions of the whole sequence at once (a matrix
        # product over the sequence); the recurrence itself is step by step
        gx = _f64(X[nb]) @ Wi + b[None, :]
        h = np.zeros(H)
        c = np.zeros(H)
        for t in range(nb.shape[0]):
            h, c = lstm_cell(gx[t] + h @ Wh, c)
        A[n] = h
    return A


def lstm_cell(z, c):
    """One LSTM step from the gate pre-activations z = [i | f | g | o]."""
    H = c.shape[0]
    i = sigmoid(z[:H])
    f = sigmoid(z[H:2 * H])
    g = np.tanh(z[2 * H:3 * H])
    o = sigmoid(z[3 * H:])
    c = f * c + i * g
    return o * np.tanh(c), c


def sage_lstm_layer(row_ptr, col_idx, X, W_ih, b_ih, W_hh, b_hh, W, b, rows=None):
    """GraphSAGE layer with the LSTM reduction (Table I, GraphSAGE row:
    LSTM(in_edges) Gather, MLP ApplyVertex; reading R8):
    y_v = [x_v | a_v] W + b with a_v = lstm_gather(...)."""
    rows = _rows_arg(rows, len(row_ptr) - 1)
    A = lstm_gather(row_ptr, col_idx, X, W_ih, b_ih, W_hh, b_hh, rows=rows)
    cat = np.concatenate([_f64(X[rows]), A], axis=1)
    return dense(cat, W, bias=b)


def sage_lstm_layer_of(g, rows=None):
    return sage_lstm_layer(g["row_ptr"], g["col_idx"], g["X"], g["W_ih"], g["b_ih"], g["W_hh"],
                           g["b_hh"], g["W"], g["b"], rows=rows)


# ==========================================================================
# R-GCN: typed edges (Table I, R-GCN row; Sec. 3.2 "ApplyEdge"; reading R9)
# ==========================================================================


def relation_counts(row_ptr, etype, num_rel, rows=None):
    """c[i, r]: number of in-edges of destination rows[i] whose type is r."""
    rp = np.asarray(row_ptr, dtype=np.int64)
    et = np.asarray(etype, dtype=np.int64)
    rows = _rows_arg(rows, rp.shape[0] - 1)
    c = np.zeros((rows.shape[0], num_rel), dtype=np.int64)
    for i, v in enumerate(rows):
        np.add.at(c[i], et[rp[v]:rp[v + 1]], 1)
    return c


def rel_gather(row_ptr, col_idx, etype, X, num_rel, rows=None):
    """Per destination v and relation r, the mean of the source rows over
    v's in-edges of type r: A[i, r] = (1 / c(v, r)) sum x_u; 0 where
    c(v, r) = 0.  Returns len(rows) x num_rel x F float64."""
    rp = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col_idx, dtype=np.int64)
    et = np.asarray(etype, dtype=np.int64)
    rows = _rows_arg(rows, rp.shape[0] - 1)
    X = np.asarray(X)
    A = np.zeros((rows.shape[0], num_rel, X.shape[1]), dtype=np.float64)
    for i, v in enumerate(rows):
        for e in range(rp[v], rp[v + 1]):
            A[i, et[e]] += _f64(X[col[e]])
    c = relation_counts(row_ptr, etype, num_rel, rows=rows)
    nz = c > 0
    A[nz] /= c[nz][:, None]
    return A


def rgcn_layer(row_ptr, col_idx, etype, X, W_rel, W_self, b, act="none", rows=None):
    """R-GCN layer, aggregate first per relation (reading R9):
    y_v = act(b + x_v W_self + sum_r A[v, r] W_r), W_rel[r] = W_r (F_in x
    F_out)."""
    rows = _rows_arg(rows, len(row_ptr) - 1)
    W_rel = _f64(W_rel)
    A = rel_gather(row_ptr, col_idx, etype, X, W_rel.shape[0], rows=rows)
    Y = dense(X[rows], W_self, bias=b)
    for r in range(W_rel.shape[0]):
        Y = Y + dense(A[:, r, :], W_rel[r])
    return ACTS[act](Y)


def rgcn_layer_of(g, rows=None):
    return rgcn_layer(g["row_ptr"], g["col_idx"], g["etype"], g["X"], g["W_rel"], g["W_self"],
                      g["b"], act=g.get("act", "none"), rows=rows)


def rel_layout(row_ptr, col_idx, etype, num_rel, tile):
    """The library's typed layout (its own definition, compared bit for bit).

    The per-edge transform x_u W_r depends only on the (relation, source)
    pair, so it is computed once per distinct pair.  Pairs are numbered
    relation by relation, sources ascending within a relation; the pair
    range of relation r starts at rel_ptr[r], a multiple of ``tile``, and is
    padded with -1 up to the next one.  Returns a dict:
      rel_count[r]  distinct sources of relation r
      rel_ptr[r]    first pair row of relation r (rel_ptr[num_rel] = total)
      pair_src[q]   source vertex of pair row q, -1 in the padding
      edge_pair[e]  pair row of CSR entry e
      edge_norm[e]  float32(1 / c(v, r)) for CSR entry e = u -> v of type r
    """
    rp = np.asarray(row_ptr, dtype=np.int64)
    col = np.asarray(col_idx, dtype=np.int64)
    et = np.asarray(etype, dtype=np.int64)
    srcs = [np.unique(col[et == r]) for r in range(num_rel)]
    rel_count = np.array([s.shape[0] for s in srcs], dtype=np.int64)
    rel_ptr = np.zeros(num_rel + 1, dtype=np.int64)
    np.cumsum((rel_count + tile - 1) // tile * tile, out=rel_ptr[1:])
    pair_src = np.full(rel_ptr[-1], -1, dtype=np.int64)
    for r in range(num_rel):
        pair_src[rel_ptr[r]:rel_ptr[r] + rel_count[r]] = srcs[r]
    edge_pair = np.zeros(col.shape[0], dtype=np.int64)
    for r in range(num_rel):
        m = et == r
        edge_pair[m] = rel_ptr[r] + np.searchsorted(srcs[r], col[m])
    c = np.zeros(col.shape[0], dtype=np.int64)
    for v in np.flatnonzero(rp[1:] > rp[:-1]):  # rows with in-edges
        t = et[rp[v]:rp[v + 1]]
        cnt = np.bincount(t, minlength=num_rel)
        c[rp[v]:rp[v + 1]] = cnt[t]
    edge_norm = np.zeros(col.shape[0], dtype=np.float32)
    nz = c > 0
    edge_norm[nz] = (1.0 / c[nz]).astype(np.float32)
    return dict(rel_count=rel_count, rel_ptr=rel_ptr, pair_src=pair_src, edge_pair=edge_pair,
                edge_norm=edge_norm)
