"""Layer and model compositions over the C ABI (torch only allocates).

``Layer`` binds a ``saga_layer_desc`` to device weights and preallocates its
workspace and output, so a forward pass enqueues kernels and nothing else.
The two-layer models of the workloads (GCN: ReLU then raw output; GAT:
concat + ELU then head mean) are sequences of such layers.
"""
from __future__ import annotations

import ctypes as C

import torch

from . import saga as S


def _dev(t, device, dtype=None):
    if t is None:
        return None
    t = torch.as_tensor(t)
    return t.to(device=device, dtype=dtype or t.dtype).contiguous()


class Layer:
    """One SAGA-NN layer (Table I model) with preallocated buffers."""

    def __init__(self, graph: S.Graph, kind: str, in_feat: int, out_feat: int, weights: dict,
                 dtype=torch.float32, act="none", heads=1, head_mean=False, neg_slope=0.2,
                 edge_feat=0, out_ld=None, hidden=0, rel=None):
        dev = graph.row_ptr.device
        self.graph = graph
        self.dtype = dtype
        wdt = dtype
        kinds = {"gcn": S.SAGA_LAYER_GCN, "gat": S.SAGA_LAYER_GAT, "sage_pool": S.SAGA_LAYER_SAGE_POOL,
                 "gated_gru": S.SAGA_LAYER_GATED_GRU, "sage_lstm": S.SAGA_LAYER_SAGE_LSTM,
                 "rgcn": S.SAGA_LAYER_RGCN}
        self.w = {k: (_dev(v, dev, wdt if k in ("w", "w_pool", "w_self") else torch.float32))
                  for k, v in weights.items()}
        d = S.saga_layer_desc()
        d.kind = kinds[kind]
        d.dtype = S.dtype_code(dtype)
        d.in_feat = in_feat
        d.out_feat = out_feat
        d.heads = heads
        d.head_mean = int(head_mean)
        d.neg_slope = neg_slope
        d.act = S.ACT[act]
        d.edge_feat = edge_feat
        d.hidden = hidden
        for k in ("w", "b", "w_pool", "b_pool", "attn_l", "attn_r", "w_e", "b_e", "w_ih", "b_ih",
                  "w_hh", "b_hh", "w_self"):
            t = self.w.get(k)
            setattr(d, k, None if t is None else t.data_ptr())
        self.rel = rel  # keeps the RelGraph (and its device arrays) alive
        if rel is not None:
            d.rel = C.pointer(rel.rel)
        self.desc = d
        self.ws_bytes = S.saga_layer_workspace_size(graph.plan, d)
        self.ws = S.workspace(self.ws_bytes, dev)
        es = torch.tensor([], dtype=dtype).element_size()
        ld = out_ld or ((out_feat * es + 15) // 16 * 16) // es
        self.out_buf = torch.empty((graph.num_dst, ld), dtype=dtype, device=dev)
        self.out = self.out_buf[:, :out_feat]

    def __call__(self, x, edge_feat=None, stream=None):
        S.saga_layer(self.graph.plan, self.desc, S.cmat(x), S.cmat(edge_feat), S.mat(self.out),
                     C.c_void_p(self.ws.data_ptr()), self.ws.numel(), S.stream_handle(stream))
        return self.out


def gcn2(graph, W1, b1, W2, b2, dtype=torch.float32, out_ld=None):
    """2-layer GCN: ReLU after layer 1, raw output after layer 2."""
    l1 = Layer(graph, "gcn", W1.shape[0], W1.shape[1], {"w": W1, "b": b1}, dtype=dtype, act="relu")
    l2 = Layer(graph, "gcn", W2.shape[0], W2.shape[1], {"w": W2, "b": b2}, dtype=dtype, act="none",
               out_ld=out_ld)
    return [l1, l2]


def gat2(graph, g, dtype=torch.float32):
    """2-layer GAT: heads concatenated + ELU, then heads averaged."""
    K = g["heads"]
    F1 = g["W1"].shape[1]
    l1 = Layer(graph, "gat", g["W1"].shape[0], F1,
               {"w": g["W1"], "b": g["b1"], "attn_l": g["al1"], "attn_r": g["ar1"]},
               heads=K, act="elu", neg_slope=g["neg_slope"])
    l2 = Layer(graph, "gat", F1, g["W2"].shape[1] // K,
               {"w": g["W2"], "b": g["b2"], "attn_l": g["al2"], "attn_r": g["ar2"]},
               heads=K, head_mean=True, act="none", neg_slope=g["neg_slope"])
    return [l1, l2]


def sage_pool(graph, g):
    F = g["W_pool"].shape[0]
    return [Layer(graph, "sage_pool", F, g["W"].shape[1],
                  {"w": g["W"], "b": g["b"], "w_pool": g["W_pool"], "b_pool": g["b_pool"]})]


def gated_gru(graph, g):
    F = g["H"].shape[1]
    return [Layer(graph, "gated_gru", F, F,
                  {"w_e": g["W_e"], "b_e": g["b_e"], "w_ih": g["W_ih"], "b_ih": g["b_ih"],
                   "w_hh": g["W_hh"], "b_hh": g["b_hh"]}, edge_feat=g["E_feat"].shape[1])]


def sage_lstm(graph, g):
    """GraphSAGE layer with the LSTM Gather: out = [x | LSTM(in-edges)] W + b."""
    F, G4 = g["W_ih"].shape
    return [Layer(graph, "sage_lstm", F, g["W"].shape[1],
                  {"w": g["W"], "b": g["b"], "w_ih": g["W_ih"], "b_ih": g["b_ih"],
                   "w_hh": g["W_hh"], "b_hh": g["b_hh"]}, hidden=G4 // 4)]


def rgcn(graph, rel, g, dtype=torch.float32):
    """R-GCN layer: act(x_v W_self + b + sum over in-edges of x_u W_r / c(v, r))."""
    R, Fi, Fo = g["W_rel"].shape
    return [Layer(graph, "rgcn", Fi, Fo,
                  {"w": g["W_rel"].reshape(R * Fi, Fo), "w_self": g["W_self"], "b": g["b"]},
                  dtype=dtype, act=g.get("act", "none"), rel=rel)]


def run(layers, x, edge_feat=None, stream=None):
    h = x
    for l in layers:
        h = l(h, edge_feat=edge_feat, stream=stream)
    return h
