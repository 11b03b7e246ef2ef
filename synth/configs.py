"""The five benchmark workloads as seeded synthetic inputs.

Each builder returns a plain dict of numpy arrays (graph as canonical
in-CSR, features, weights).  Seeds: ``SeedSequence(200900804,
spawn_key=(K, s))`` with s = 0 graph, 1 vertex features, 2 edge features,
3 weights, 4 relabelling permutation, 5 equivariance permutation.  Scaled
test variants use K + 100.

Workloads (the paper's dataset shapes are stood in for by these graphs):
  gcn_er      2-layer GCN, Erdos-Renyi 2,000 vertices, 10,000 directed edges
              + self-loops, features 128 binary (5 % ones), 128->16->8.
  gat_ba      2-layer GAT 8 heads x 8 dims, Barabasi-Albert 20,000 vertices,
              m = 5, symmetrised + self-loops, features 512 N(0,1).
  sage_rmat   GraphSAGE-pool, R-MAT (0.57, 0.19, 0.19) scale 17, 16 edges per
              vertex, relabelled, features 256 N(0,1).
  gated_rgg   gated edge MPNN + GRU, torus random geometric graph 100,000
              vertices, expected degree 12, h 64-d, e 16-d N(0,1).
  gcn_rmat    2-layer GCN, R-MAT scale 21, 50 edges per vertex, relabelled
              + self-loops, features 602 N(0,1), 602->128->41, float32 and
              bfloat16 storage variants.
  sage_lstm   GraphSAGE with the LSTM Gather on the sage_rmat graph and
              features, hidden 128, output 256.
  rgcn_rmat   R-GCN layer (typed edges), R-MAT scale 18, 16 edges per
              vertex, relabelled, 32 relation types drawn per edge with
              P(r) proportional to 1/(r+1), features 128 N(0,1) -> 64, ReLU.
"""
from __future__ import annotations

import math

import numpy as np

from . import graphs as G
from . import tensors as T

RMAT_ABC = (0.57, 0.19, 0.19)


def _csr_dict(name, n, src, dst, want_eid=False):
    res = G.to_in_csr(n, src, dst, want_eid=want_eid)
    d = {"name": name, "num_vertices": n, "row_ptr": res[0], "col_idx": res[1]}
    if want_eid:
        d["eid"] = res[2]
    d["num_edges"] = int(res[1].shape[0])
    return d


# --------------------------------------------------------------------------
def gcn_er(n=2000, m=10000, f_in=128, hidden=16, f_out=8, key=1):
    src, dst = G.er_directed(n, m, G.rng_for(key, 0))
    src, dst = G.add_self_loops(src, dst, n)
    d = _csr_dict("gcn_er", n, src, dst)
    d["model"] = "gcn"
    d["X"] = T.sparse_binary_matrix(n, f_in, 0.05, G.rng_for(key, 1))
    rw = G.rng_for(key, 3)
    d["W1"] = T.glorot(f_in, hidden, rw)
    d["b1"] = T.bias(f_in, hidden, rw)
    d["W2"] = T.glorot(hidden, f_out, rw)
    d["b2"] = T.bias(hidden, f_out, rw)
    d["dims"] = (f_in, hidden, f_out)
    return d


def gat_ba(n=20000, m=5, f_in=512, heads=8, head_dim=8, key=2):
    src, dst = G.ba_undirected(n, m, G.rng_for(key, 0))
    src, dst = G.symmetrise(src, dst)
    src, dst = G.add_self_loops(src, dst, n)
    d = _csr_dict("gat_ba", n, src, dst)
    d["model"] = "gat"
    d["X"] = T.normal_matrix(n, f_in, (key, 1))
    rw = G.rng_for(key, 3)
    F = heads * head_dim
    d["W1"] = T.glorot(f_in, F, rw)
    d["al1"] = T.glorot(head_dim, 1, rw, shape=(heads, head_dim))
    d["ar1"] = T.glorot(head_dim, 1, rw, shape=(heads, head_dim))
    d["b1"] = T.bias(f_in, F, rw)
    d["W2"] = T.glorot(F, F, rw)
    d["al2"] = T.glorot(head_dim, 1, rw, shape=(heads, head_dim))
    d["ar2"] = T.glorot(head_dim, 1, rw, shape=(heads, head_dim))
    d["b2"] = T.bias(F, head_dim, rw)
    d["heads"] = heads
    d["head_dim"] = head_dim
    d["neg_slope"] = 0.2
    return d


def sage_rmat(scale=17, avg_deg=16, f=256, key=3):
    n = 1 << scale
    E = avg_deg * n
    src, dst = G.rmat(scale, E, *RMAT_ABC, key=(key, 0))
    perm = G.rng_for(key, 4).permutation(n).astype(np.int32)
    src, dst = G.relabel(src, dst, perm)
    d = _csr_dict("sage_rmat", n, src, dst)
    d["model"] = "sage_pool"
    d["X"] = T.normal_matrix(n, f, (key, 1))
    rw = G.rng_for(key, 3)
    d["W_pool"] = T.glorot(f, f, rw)
    d["b_pool"] = T.bias(f, f, rw)
    d["W"] = T.glorot(2 * f, f, rw)
    d["b"] = T.bias(2 * f, f, rw)
    return d


def sage_lstm(scale=17, avg_deg=16, f=256, hidden=128, f_out=256, key=6, graph_key=3):
    """GraphSAGE with the LSTM Gather on the GraphSAGE-pool workload's R-MAT
    graph and features (same graph_key); LSTM weights U(+-1/sqrt(hidden))."""
    n = 1 << scale
    E = avg_deg * n
    src, dst = G.rmat(scale, E, *RMAT_ABC, key=(graph_key, 0))
    perm = G.rng_for(graph_key, 4).permutation(n).astype(np.int32)
    src, dst = G.relabel(src, dst, perm)
    d = _csr_dict("sage_lstm", n, src, dst)
    d["model"] = "sage_lstm"
    d["X"] = T.normal_matrix(n, f, (graph_key, 1))
    rw = G.rng_for(key, 3)
    a = 1.0 / np.sqrt(hidden)
    d["W_ih"] = rw.uniform(-a, a, (f, 4 * hidden)).astype(np.float32)
    d["W_hh"] = rw.uniform(-a, a, (hidden, 4 * hidden)).astype(np.float32)
    d["b_ih"] = rw.uniform(-a, a, 4 * hidden).astype(np.float32)
    d["b_hh"] = rw.uniform(-a, a, 4 * hidden).astype(np.float32)
    d["W"] = T.glorot(f + hidden, f_out, rw)
    d["b"] = T.bias(f + hidden, f_out, rw)
    d["dims"] = (f, hidden, f_out)
    return d


def gated_rgg(n=100000, avg_deg=12, f=64, fe=16, key=4):
    r = math.sqrt(avg_deg / (math.pi * (n - 1)))
    src, dst = G.torus_rgg(n, r, G.rng_for(key, 0))
    src, dst = G.symmetrise(src, dst)
    d = _csr_dict("gated_rgg", n, src, dst)
    d["model"] = "gated_gru"
    d["radius"] = r
    d["H"] = T.normal_matrix(n, f, (key, 1))
    # one 16-d feature row per directed edge, stored in CSR order
    d["E_feat"] = T.normal_matrix(d["num_edges"], fe, (key, 2))
    rw = G.rng_for(key, 3)
    d["W_e"] = T.glorot(2 * f + fe, f, rw)
    d["b_e"] = T.bias(2 * f + fe, f, rw)
    d["W_ih"] = T.glorot(f, 3 * f, rw)
    d["b_ih"] = T.bias(f, 3 * f, rw)
    d["W_hh"] = T.glorot(f, 3 * f, rw)
    d["b_hh"] = T.bias(f, 3 * f, rw)
    return d


def gcn_rmat(scale=21, avg_deg=50, f_in=602, hidden=128, f_out=41, key=5,
             bf16=False):
    n = 1 << scale
    E = avg_deg * n
    src, dst = G.rmat(scale, E, *RMAT_ABC, key=(key, 0))
    perm = G.rng_for(key, 4).permutation(n).astype(np.int32)
    src, dst = G.relabel(src, dst, perm)
    src, dst = G.add_self_loops(src, dst, n)
    d = _csr_dict("gcn_rmat", n, src, dst)
    del src, dst
    d["model"] = "gcn"
    ld = f_in + (-f_in) % 4  # 16-byte rows in float32
    d["X"] = T.normal_matrix(n, f_in, (key, 1), ld=ld)
    rw = G.rng_for(key, 3)
    d["W1"] = T.glorot(f_in, hidden, rw)
    d["b1"] = T.bias(f_in, hidden, rw)
    d["W2"] = T.glorot(hidden, f_out, rw)
    d["b2"] = T.bias(hidden, f_out, rw)
    d["dims"] = (f_in, hidden, f_out)
    if bf16:
        add_bf16_variant(d)
    return d


def rgcn_rmat(scale=18, avg_deg=16, num_rel=32, f_in=128, f_out=64, key=7):
    """R-GCN layer on a typed power-law graph.  The edge type (stream 2, the
    edge-attribute stream) is drawn per edge, independently of its
    endpoints, with P(r) proportional to 1 / (r + 1); ``etype`` is aligned
    with the CSR entries."""
    n = 1 << scale
    E = avg_deg * n
    src, dst = G.rmat(scale, E, *RMAT_ABC, key=(key, 0))
    perm = G.rng_for(key, 4).permutation(n).astype(np.int32)
    src, dst = G.relabel(src, dst, perm)
    p = 1.0 / np.arange(1, num_rel + 1, dtype=np.float64)
    et = G.rng_for(key, 2).choice(num_rel, E, p=p / p.sum()).astype(np.int32)
    d = _csr_dict("rgcn_rmat", n, src, dst, want_eid=True)
    d["etype"] = et[d.pop("eid")]
    d["model"] = "rgcn"
    d["num_rel"] = num_rel
    d["X"] = T.normal_matrix(n, f_in, (key, 1))
    rw = G.rng_for(key, 3)
    d["W_rel"] = np.stack([T.glorot(f_in, f_out, rw) for _ in range(num_rel)])
    d["W_self"] = T.glorot(f_in, f_out, rw)
    d["b"] = T.bias(f_in, f_out, rw)
    d["act"] = "relu"
    d["dims"] = (f_in, f_out)
    return d


def add_bf16_variant(d):
    """bfloat16 storage of X and the weights (round to nearest even); the
    float32 arrays ``X_bf``, ``W1_bf``, ``W2_bf`` hold their exact values."""
    f_in = d["dims"][0]
    ld = f_in + (-f_in) % 8  # 16-byte rows in bfloat16
    d["X_bf16"] = T.bf16_padded_from_f32(d["X"], f_in, ld)
    d["W1_bf16"] = T.bf16_bits(d["W1"])
    d["W2_bf16"] = T.bf16_bits(d["W2"])
    d["W1_bf"] = T.bf16_to_f32(d["W1_bf16"])
    d["W2_bf"] = T.bf16_to_f32(d["W2_bf16"])
    return d


BUILDERS = {
    "gcn_er": gcn_er,
    "gat_ba": gat_ba,
    "sage_rmat": sage_rmat,
    "gated_rgg": gated_rgg,
    "gcn_rmat": gcn_rmat,
    "sage_lstm": sage_lstm,
    "rgcn_rmat": rgcn_rmat,
}

# scaled variants used by parity tests (K + 100 seeds)
SMALL = {
    "gcn_er": dict(key=101),
    "gat_ba": dict(n=3000, key=102),
    "sage_rmat": dict(scale=12, key=103),
    "gated_rgg": dict(n=8000, key=104),
    "gcn_rmat": dict(scale=13, avg_deg=50, key=105),
    "sage_lstm": dict(scale=10, key=106, graph_key=106),
    "rgcn_rmat": dict(scale=11, key=107),
}


def build(name: str, small: bool = False, **kw):
    args = dict(SMALL[name]) if small else {}
    args.update(kw)
    return BUILDERS[name](**args)
