"""R-GCN on the GPU against the oracle (Table I, R-GCN row; Sec. 3.2
"ApplyEdge"): the typed layout bit for bit, the grouped per-relation
transform, the typed Gather with the self term, and the whole layer, in
float32 and bfloat16, on tiny typed multigraphs, relations without edges,
an edgeless graph, a hub row split over several segments, and the full
2^18-vertex workload on sampled rows."""
import ctypes as C

import numpy as np
import pytest
import torch

from gpu_util import dev_int, dev_padded, device, lib, to_np
from helpers import BF16_TOL, FP32_TOL, edges_to_csr, rel_err, tiny_graphs
from oracle import saga_oracle as O
from synth import tensors as T

pytestmark = pytest.mark.gpu
TILE = 128


def _typed_cases():
    out = []
    rng = np.random.default_rng(21)
    for name, n, src, dst in tiny_graphs():
        R = 3
        types = rng.integers(0, R, len(src)).tolist()
        rp, col, order = edges_to_csr(n, src, dst)
        et = np.array([types[e] for e in order], np.int32)
        out.append((name, n, R, rp, col, et))
    # relations 1 and 4 carry no edge; one relation with exactly TILE sources
    n = 400
    src = list(range(TILE)) + rng.integers(0, n, 900).tolist()
    dst = rng.integers(0, n, len(src)).tolist()
    types = [2] * TILE + rng.choice([0, 3, 5], 900).tolist()
    rp, col, order = edges_to_csr(n, src, dst)
    out.append(("gaps", n, 6, rp, col, np.array([types[e] for e in order], np.int32)))
    # a hub row of 3000 in-edges (split over several segments) with 7 types
    n = 300
    d = np.zeros(n, np.int64)
    d[5], d[6] = 3000, 40
    d[10:100] = rng.integers(1, 12, 90)
    rp = np.concatenate([[0], np.cumsum(d)]).astype(np.int32)
    E = int(rp[-1])
    col = np.sort(rng.integers(0, n, E).reshape(-1)).astype(np.int32)
    for v in range(n):
        col[rp[v]:rp[v + 1]] = np.sort(col[rp[v]:rp[v + 1]])
    out.append(("hub", n, 7, rp, col, rng.integers(0, 7, E).astype(np.int32)))
    from synth import configs as Cfg

    g = Cfg.build("rgcn_rmat", small=True)
    out.append(("rmat", g["num_vertices"], g["num_rel"], g["row_ptr"], g["col_idx"], g["etype"]))
    return out


CASES = _typed_cases()


def _rel(n, R, rp, col, et, seg_len=0):
    S = lib()
    graph = S.Graph(dev_int(rp), dev_int(col), seg_len=seg_len)
    return graph, S.RelGraph(graph, dev_int(et), R)


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_rel_layout_bit_exact(case):
    name, n, R, rp, col, et = case
    print(f"rel layout {name}", flush=True)
    graph, rg = _rel(n, R, rp, col, et)
    want = O.rel_layout(rp, col, et, R, TILE)
    got = {k: v.cpu().numpy() for k, v in rg.arrays().items()}
    assert rg.counts.pair_rows == want["rel_ptr"][-1]
    assert rg.counts.pairs == want["rel_count"].sum()
    for k in ("rel_ptr", "rel_count", "pair_src", "edge_pair"):
        assert np.array_equal(got[k].astype(np.int64), want[k]), k
    assert np.array_equal(got["edge_norm"].view(np.uint32), want["edge_norm"].view(np.uint32))


def test_rel_layout_edgeless_and_single_relation():
    n = 50
    rp = np.zeros(n + 1, np.int32)
    graph, rg = _rel(n, 1, rp, np.zeros(0, np.int32), np.zeros(0, np.int32))
    assert rg.counts.pair_rows == 0 and rg.counts.pairs == 0
    name, n, R, rp, col, et = CASES[0]
    graph, rg = _rel(n, 1, rp, col, np.zeros_like(et))
    want = O.rel_layout(rp, col, np.zeros_like(et), 1, TILE)
    got = rg.arrays()
    assert np.array_equal(got["pair_src"].cpu().numpy(), want["pair_src"])
    assert np.array_equal(got["edge_pair"].cpu().numpy(), want["edge_pair"])


def test_rel_plan_flags_out_of_range_types():
    S = lib()
    name, n, R, rp, col, et = CASES[0]
    bad = et.copy()
    bad[3] = R  # outside [0, R)
    graph = S.Graph(dev_int(rp), dev_int(col))
    rg = S.RelGraph(graph, dev_int(bad), R, check=False)
    st, counts = S.saga_rel_plan_check(rg.rel, S.stream_handle())
    assert st == S.SAGA_EGRAPH and counts.error_flags == 1
    # every later call on this rel plan leaves its output unwritten
    F = 8
    src = dev_padded(np.ones((rg.rel.max_pairs, F)))
    out = dev_padded(np.zeros((n, F)), fill=7.0)
    out.fill_(7.0)
    op = S.saga_edge_op(S.SAGA_MSG_TYPED, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 0, 0.0, 0)
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(src)
    inp.rel = C.pointer(rg.rel)
    ws = S.workspace(S.saga_gather_workspace_size(graph.plan, op, F), device())
    S.saga_scatter_apply_edge_gather(graph.plan, op, inp, S.mat(out), C.c_void_p(ws.data_ptr()),
                                     ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())


def _run_transform(rg, X, W, dtype):
    S = lib()
    R, K, N = W.shape
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    code = S.SAGA_F32 if dtype == "f32" else S.SAGA_BF16
    if dtype == "f32":
        x = dev_padded(X)
        w = torch.from_numpy(np.ascontiguousarray(W.reshape(R * K, N), np.float32)).to(device())
    else:
        x = dev_padded(X, dtype=torch.bfloat16)
        w = torch.from_numpy(W.reshape(R * K, N).astype(np.float32)).to(device()).to(torch.bfloat16)
    out = torch.full((rg.rel.max_pairs, N), float("nan"), dtype=tdt, device=device())
    ws = S.workspace(S.saga_rel_transform_workspace_size(rg.rel, code, K, N), device())
    S.saga_rel_transform(rg.rel, code, S.cmat(x), S.cmat(w), S.mat(out), C.c_void_p(ws.data_ptr()),
                         ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    return to_np(out)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("kn", [(32, 16), (100, 41), (128, 64), (64, 200)], ids=str)
@pytest.mark.parametrize("case", [CASES[3], CASES[4], CASES[6]], ids=lambda c: c[0])
def test_rel_transform_matches_oracle(case, kn, dtype):
    name, n, R, rp, col, et = case
    K, N = kn
    print(f"rel transform {name} K={K} N={N} {dtype}", flush=True)
    graph, rg = _rel(n, R, rp, col, et)
    rng = np.random.default_rng(K * N)
    X = rng.standard_normal((n, K)).astype(np.float32)
    W = rng.standard_normal((R, K, N)).astype(np.float32) / np.sqrt(K)
    if dtype == "bf16":  # the exact bfloat16 values both sides see
        X = T.bf16_to_f32(T.bf16_bits(X))
        W = T.bf16_to_f32(T.bf16_bits(W))
    got = _run_transform(rg, X, W, dtype)
    L = O.rel_layout(rp, col, et, R, TILE)
    rows = int(L["rel_ptr"][-1])
    want = np.zeros((rows, N))
    for r in range(R):
        q0, q1 = L["rel_ptr"][r], L["rel_ptr"][r] + L["rel_count"][r]
        want[q0:q1] = O.dense(X[L["pair_src"][q0:q1]], W[r])
    pad = L["pair_src"] < 0
    assert np.all(got[:rows][pad] == 0.0)
    assert rel_err(got[:rows][~pad], want[~pad]) <= (FP32_TOL if dtype == "f32" else BF16_TOL)


def test_rel_transform_exact_on_small_integers():
    name, n, R, rp, col, et = CASES[4]
    graph, rg = _rel(n, R, rp, col, et)
    rng = np.random.default_rng(3)
    X = rng.integers(-3, 4, (n, 40)).astype(np.float32)
    W = rng.integers(-2, 3, (R, 40, 24)).astype(np.float32)
    got = _run_transform(rg, X, W, "f32")
    L = O.rel_layout(rp, col, et, R, TILE)
    for r in range(R):
        q0, q1 = L["rel_ptr"][r], L["rel_ptr"][r] + L["rel_count"][r]
        assert np.array_equal(got[q0:q1], X[L["pair_src"][q0:q1]].astype(np.float64) @ W[r])


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_typed_gather_with_self_matches_oracle(case, dtype):
    """out_v = act(self_v + b + sum_e norm_e src[pair_e]) on given pair rows."""
    S = lib()
    name, n, R, rp, col, et = case
    print(f"typed gather {name} {dtype}", flush=True)
    graph, rg = _rel(n, R, rp, col, et, seg_len=64)
    F = 24
    rng = np.random.default_rng(5)
    P = rng.standard_normal((rg.rel.max_pairs, F)).astype(np.float32)
    SELF = rng.standard_normal((n, F)).astype(np.float32)
    b = rng.standard_normal(F).astype(np.float32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    if dtype == "bf16":
        P, SELF = T.bf16_to_f32(T.bf16_bits(P)), T.bf16_to_f32(T.bf16_bits(SELF))
    src, self_t = dev_padded(P, dtype=tdt), dev_padded(SELF, dtype=tdt)
    bias = torch.from_numpy(b).to(device())
    out = dev_padded(np.zeros((n, F)), dtype=tdt)
    op = S.saga_edge_op(S.SAGA_MSG_TYPED, S.SAGA_RED_SUM, S.dtype_code(tdt), 1, 0, 0, 0.0,
                        S.SAGA_ACT_RELU)
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(src)
    inp.rel = C.pointer(rg.rel)
    inp.self = S.cmat(self_t)
    inp.bias = bias.data_ptr()
    ws = S.workspace(S.saga_gather_workspace_size(graph.plan, op, F), device())
    S.saga_scatter_apply_edge_gather(graph.plan, op, inp, S.mat(out), C.c_void_p(ws.data_ptr()),
                                     ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    L = O.rel_layout(rp, col, et, R, TILE)
    agg = np.zeros((n, F))
    for v in range(n):
        for e in range(rp[v], rp[v + 1]):
            agg[v] += np.float64(L["edge_norm"][e]) * P[L["edge_pair"][e]]
    want = O.relu(agg + SELF + b[None, :])
    assert rel_err(to_np(out), want) <= (FP32_TOL if dtype == "f32" else BF16_TOL)


def _layer(n, R, rp, col, et, g, dtype="f32"):
    from paper_2009_00804_amd import layers as LY

    graph, rg = _rel(n, R, rp, col, et)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    model = LY.rgcn(graph, rg, g, dtype=tdt)
    x = dev_padded(g["X"], dtype=tdt)
    y = LY.run(model, x)
    torch.cuda.synchronize()
    return to_np(y), (graph, rg, model, x)


def _weights(R, Fi, Fo, seed):
    rng = np.random.default_rng(seed)
    return dict(W_rel=(rng.standard_normal((R, Fi, Fo)) / np.sqrt(Fi)).astype(np.float32),
                W_self=(rng.standard_normal((Fi, Fo)) / np.sqrt(Fi)).astype(np.float32),
                b=rng.standard_normal(Fo).astype(np.float32) * 0.1, act="relu")


@pytest.mark.parametrize("case", CASES, ids=lambda c: c[0])
def test_rgcn_layer_matches_oracle(case):
    name, n, R, rp, col, et = case
    print(f"rgcn layer {name}", flush=True)
    g = _weights(R, 20, 36, 9)
    g["X"] = np.random.default_rng(1).standard_normal((n, 20)).astype(np.float32)
    got, _ = _layer(n, R, rp, col, et, g)
    want = O.rgcn_layer(rp, col, et, g["X"], g["W_rel"], g["W_self"], g["b"], act="relu")
    assert rel_err(got, want) <= FP32_TOL


def test_rgcn_layer_bf16():
    name, n, R, rp, col, et = CASES[-1]
    g = _weights(R, 64, 32, 4)
    X = np.random.default_rng(2).standard_normal((n, 64)).astype(np.float32)
    bf = lambda a: T.bf16_to_f32(T.bf16_bits(a))  # noqa: E731
    g["X"], g["W_rel"], g["W_self"] = bf(X), bf(g["W_rel"]), bf(g["W_self"])
    got, _ = _layer(n, R, rp, col, et, g, dtype="bf16")
    want = O.rgcn_layer(rp, col, et, g["X"], g["W_rel"], g["W_self"], g["b"], act="relu")
    assert rel_err(got, want) <= BF16_TOL


def test_rgcn_layer_edgeless_graph_is_self_term():
    n, R = 70, 3
    rp = np.zeros(n + 1, np.int32)
    g = _weights(R, 16, 8, 3)
    g["X"] = np.random.default_rng(0).standard_normal((n, 16)).astype(np.float32)
    got, _ = _layer(n, R, rp, np.zeros(0, np.int32), np.zeros(0, np.int32), g)
    assert rel_err(got, O.dense(g["X"], g["W_self"], bias=g["b"], act="relu")) <= FP32_TOL


def test_rgcn_layer_deterministic():
    name, n, R, rp, col, et = CASES[-2]
    g = _weights(R, 32, 48, 6)
    g["X"] = np.random.default_rng(3).standard_normal((n, 32)).astype(np.float32)
    from paper_2009_00804_amd import layers as LY

    a, (graph, rg, model, x) = _layer(n, R, rp, col, et, g)
    b = to_np(LY.run(model, x))
    torch.cuda.synchronize()
    assert np.array_equal(a, b)


@pytest.mark.slow
def test_rgcn_full_workload_sampled():
    """The 2^18-vertex, 32-relation workload in the configuration the
    benchmark times; the oracle evaluates sampled rows, the hubs included."""
    from synth import configs as Cfg

    g = Cfg.build("rgcn_rmat")
    n, R = g["num_vertices"], g["num_rel"]
    print(f"rgcn full V={n} E={g['num_edges']}", flush=True)
    got, (graph, rg, model, x) = _layer(n, R, g["row_ptr"], g["col_idx"], g["etype"], g)
    d = np.diff(g["row_ptr"].astype(np.int64))
    rng = np.random.default_rng(0)
    rows = np.unique(np.concatenate([np.argsort(d)[-4:], rng.integers(0, n, 40),
                                     np.flatnonzero(d == 0)[:3]]))
    want = O.rgcn_layer_of(g, rows=rows)
    assert rel_err(got[rows], want) <= FP32_TOL
    assert np.isfinite(got).all()
    # the layout of the whole graph, bit for bit
    L = O.rel_layout(g["row_ptr"], g["col_idx"], g["etype"], R, TILE)
    arr = {k: v.cpu().numpy() for k, v in rg.arrays().items()}
    for k in ("rel_ptr", "pair_src", "edge_pair"):
        assert np.array_equal(arr[k].astype(np.int64), L[k]), k
    assert np.array_equal(arr["edge_norm"], L["edge_norm"])


def test_rel_layout_bitmap_atomics_path():
    """Many sources x many relations: the pair bitmap is set with atomics
    instead of byte flags (R x 32 W bytes above 256 MB); same layout."""
    n, R, E = 1 << 21, 200, 60000
    rng = np.random.default_rng(17)
    src = rng.integers(0, n, E)
    dst = np.sort(rng.integers(0, n, E))
    # hub sources and hub destinations with repeated types as well
    src[:5000] = 7
    dst[-4000:] = n - 3
    order = np.lexsort((src, dst))
    src, dst = src[order], dst[order]
    rp = np.zeros(n + 1, np.int64)
    np.cumsum(np.bincount(dst, minlength=n), out=rp[1:])
    et = rng.integers(0, R, E).astype(np.int32)
    et[:5000] = rng.integers(0, 3, 5000)
    print(f"rel layout bitmap path V={n} E={E} R={R}", flush=True)
    graph, rg = _rel(n, R, rp.astype(np.int32), src.astype(np.int32), et)
    want = O.rel_layout(rp, src, et, R, TILE)
    got = {k: v.cpu().numpy() for k, v in rg.arrays().items()}
    for k in ("rel_ptr", "rel_count", "pair_src", "edge_pair"):
        assert np.array_equal(got[k].astype(np.int64), want[k]), k
    assert np.array_equal(got["edge_norm"], want["edge_norm"])
