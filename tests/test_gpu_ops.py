"""Op-level parity of the HIP kernels against the CPU oracle: the fused
Scatter+ApplyEdge+Gather for every reduction and message kind, and the
ApplyVertex GEMM with its epilogues, on seeded inputs that span several
tiles, a ragged tail, empty rows and split (long) rows."""
import ctypes as C

import numpy as np
import pytest
import torch

from gpu_util import dev_padded, device, graph, lib, to_np
from helpers import BF16_TOL, FP32_TOL, edges_to_csr, rel_err, rel_err_terms, tiny_graphs
from oracle import saga_oracle as O

pytestmark = pytest.mark.gpu

ACTS = {"none": 0, "relu": 1, "elu": 2, "sigmoid": 3, "tanh": 4}


def _power_law(seed=0):
    """R-MAT graph with many empty rows and hub rows longer than seg_len."""
    from synth import configs as C_

    g = C_.build("sage_rmat", small=True)
    return g["row_ptr"], g["col_idx"], g["num_vertices"]


def _bf16_round(a):
    from synth import tensors as T

    return T.bf16_to_f32(T.bf16_bits(np.asarray(a, np.float32)))


def run_gather(g, src_t, op_kw, out_cols, out_dtype, el=None, er=None, bias=None, extra=None):
    S = lib()
    op = S.saga_edge_op()
    op.msg = op_kw.get("msg", S.SAGA_MSG_COPY)
    op.reduce = op_kw["reduce"]
    op.dtype = S.dtype_code(src_t.dtype)
    op.heads = op_kw.get("heads", 1)
    op.head_mean = op_kw.get("head_mean", 0)
    op.dst_norm = op_kw.get("dst_norm", 0)
    op.neg_slope = op_kw.get("neg_slope", 0.2)
    op.act = ACTS[op_kw.get("act", "none")]
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(src_t)
    inp.el = S.cmat(el)
    inp.er = S.cmat(er)
    if extra:
        for k, v in extra.items():
            setattr(inp, k, v)
    bias_t = None
    if bias is not None:
        bias_t = torch.from_numpy(np.asarray(bias, np.float32)).to(device())
        inp.bias = bias_t.data_ptr()
    out = dev_padded(np.zeros((g.num_dst, out_cols)), dtype=out_dtype, fill=7.0)
    n = S.saga_gather_workspace_size(g.plan, op, src_t.shape[1])
    ws = S.workspace(n, device())
    S.saga_scatter_apply_edge_gather(g.plan, op, inp, S.mat(out), C.c_void_p(ws.data_ptr()),
                                     ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    return out


def _ref_simple(rp, col, X, reduce, msg, dst_norm, bias, act, nsrc):
    d_out = O.out_degrees(col, nsrc)
    scale = O.degree_scale(d_out) if msg == "src_norm" else None
    r = O.gather(rp, col, X, reduce, src_scale=scale)
    if dst_norm:
        r = r * O.degree_scale(O.in_degrees(rp))[:, None]
    if bias is not None:
        r = r + np.asarray(bias, np.float64)[None, :]
    return O.ACTS[act](r)


GRAPHS = {"tiny_" + c[0]: c for c in tiny_graphs()}


def _get_graph(name, seg_len=16, block_cost=128):
    if name == "rmat":
        rp, col, n = _power_law()
    elif name == "edgeless":  # every row empty: the Gather output is act(bias)
        n = 37
        rp, col = np.zeros(n + 1, np.int32), np.zeros(0, np.int32)
    else:
        _, n, src, dst = GRAPHS[name]
        rp, col, _ = edges_to_csr(n, src, dst)
    return rp, col, n, graph(rp, col, num_src=n, seg_len=seg_len, block_cost=block_cost, row_cost=4)


@pytest.mark.parametrize("gname", ["rmat", "tiny_multi", "tiny_star", "tiny_random"])
@pytest.mark.parametrize("F", [1, 8, 16, 41, 64, 128, 256, 300])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gather_sum_mean(gname, F, dtype):
    S = lib()
    rp, col, n, g = _get_graph(gname)
    rng = np.random.default_rng(F)
    X = rng.standard_normal((n, F)).astype(np.float32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    if dtype == "bf16":
        X = _bf16_round(X)
    Xt = dev_padded(X, tdt)
    tol = FP32_TOL if dtype == "f32" else BF16_TOL
    bias = rng.standard_normal(F)
    cases = [
        ("sum", "copy", 0, None, "none"),
        ("sum", "src_norm", 1, bias, "relu"),
        ("mean", "copy", 0, bias, "tanh"),
    ]
    for red, msg, dn, b, act in cases:
        print(f"gather {gname} F={F} {dtype} {red} {msg} dst_norm={dn} act={act}", flush=True)
        out = run_gather(g, Xt, dict(reduce={"sum": S.SAGA_RED_SUM, "mean": S.SAGA_RED_MEAN}[red],
                                     msg={"copy": S.SAGA_MSG_COPY, "src_norm": S.SAGA_MSG_SRC_NORM}[msg],
                                     dst_norm=dn, act=act), F, tdt, bias=b)
        ref = _ref_simple(rp, col, X, red, msg, dn, b, act, n)
        got = to_np(out)
        err = rel_err(got, ref)
        assert err <= tol, (red, msg, err)
        # element by element, against the magnitude of each output's own terms
        mag = _ref_simple(rp, col, np.abs(X), red, msg, dn, None if b is None else np.abs(b), "none", n)
        err_t = rel_err_terms(got, ref, mag)
        assert err_t <= tol, (red, msg, err_t)


@pytest.mark.parametrize("gname", ["rmat", "tiny_multi", "tiny_star"])
@pytest.mark.parametrize("F", [4, 41, 128, 256])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gather_max_bit_exact(gname, F, dtype):
    S = lib()
    rp, col, n, g = _get_graph(gname)
    rng = np.random.default_rng(100 + F)
    X = rng.standard_normal((n, F)).astype(np.float32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    if dtype == "bf16":
        X = _bf16_round(X)
    print(f"gather max {gname} F={F} {dtype}", flush=True)
    out = run_gather(g, dev_padded(X, tdt), dict(reduce=S.SAGA_RED_MAX), F, tdt)
    ref = O.gather(rp, col, X, "max")
    got = to_np(out)
    assert np.array_equal(got, ref)   # exact: the max is one of the inputs (0 for empty rows)


@pytest.mark.parametrize("gname", ["rmat", "tiny_multi", "tiny_random"])
@pytest.mark.parametrize("heads,D,head_mean", [(8, 8, 0), (8, 8, 1), (2, 4, 0), (4, 16, 1), (1, 4, 0)])
def test_gather_attention(gname, heads, D, head_mean):
    S = lib()
    rp, col, n, g = _get_graph(gname)
    rng = np.random.default_rng(7 * heads + D)
    F = heads * D
    Zx = rng.standard_normal((n, F + 2 * heads)).astype(np.float32)
    Z = Zx[:, :F]
    el = Zx[:, F:F + heads]
    er = Zx[:, F + heads:]
    zt = dev_padded(Zx, torch.float32)
    bias = rng.standard_normal(D if head_mean else F)
    print(f"gather attention {gname} H={heads} D={D} mean={head_mean}", flush=True)
    out = run_gather(g, zt[:, :F], dict(msg=S.SAGA_MSG_GAT, reduce=S.SAGA_RED_SOFTMAX, heads=heads,
                                        head_mean=head_mean, act="elu", neg_slope=0.2),
                     D if head_mean else F, torch.float32, el=zt[:, F:F + heads],
                     er=zt[:, F + heads:], bias=bias)
    o = O.attention_gather(rp, col, Z, el, er, heads, 0.2)
    if head_mean:
        o = o.reshape(n, heads, D).mean(axis=1)
    ref = O.elu(o + bias[None, :])
    assert rel_err(to_np(out), ref) <= FP32_TOL


def test_concurrent_calls_from_two_threads():
    """Two host threads, each with its own stream and workspace, run Gathers
    of different widths and reductions at the same time: each result equals
    the same call made alone, byte for byte (no shared host state in the
    launch path)."""
    import threading

    S = lib()
    rp, col, n, g = _get_graph("rmat")
    rng = np.random.default_rng(31)
    X = {F: dev_padded(rng.standard_normal((n, F)).astype(np.float32)) for F in (32, 100)}
    jobs = [(32, S.SAGA_RED_SUM), (100, S.SAGA_RED_MAX), (32, S.SAGA_RED_MEAN), (100, S.SAGA_RED_SUM)]

    def run(F, red, stream):
        op = S.saga_edge_op()
        op.msg, op.reduce, op.dtype, op.heads = S.SAGA_MSG_COPY, red, S.SAGA_F32, 1
        inp = S.saga_edge_inputs()
        inp.src = S.cmat(X[F])
        out = dev_padded(np.zeros((n, F)), fill=7.0)
        ws = S.workspace(S.saga_gather_workspace_size(g.plan, op, F), device())
        sh = S.stream_handle(stream)
        for _ in range(5):
            S.saga_scatter_apply_edge_gather(g.plan, op, inp, S.mat(out), C.c_void_p(ws.data_ptr()),
                                             ws.numel(), sh)
        S.saga_sync_check(sh)
        return to_np(out)

    alone = [run(F, red, torch.cuda.current_stream()) for F, red in jobs]
    got = [None] * len(jobs)
    streams = [torch.cuda.Stream() for _ in jobs]
    torch.cuda.synchronize()

    def worker(k):
        for i in range(k, len(jobs), 2):
            got[i] = run(*jobs[i], streams[i])

    print("concurrent gathers from two threads", flush=True)
    th = [threading.Thread(target=worker, args=(k,)) for k in range(2)]
    for t in th:
        t.start()
    for t in th:
        t.join()
    for i in range(len(jobs)):
        assert got[i] is not None and np.array_equal(got[i], alone[i]), i


def test_sync_check_after_work_on_a_stream():
    """saga_sync_check waits for a side stream's work (a Gather enqueued
    there) and reports no device error; the output is then complete."""
    S = lib()
    rp, col, n, g = _get_graph("rmat")
    X = np.random.default_rng(2).standard_normal((n, 32)).astype(np.float32)
    Xt = dev_padded(X)
    side = torch.cuda.Stream()
    op = S.saga_edge_op()
    op.msg, op.reduce, op.dtype, op.heads = S.SAGA_MSG_COPY, S.SAGA_RED_SUM, S.SAGA_F32, 1
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(Xt)
    out = dev_padded(np.zeros((n, 32)), fill=7.0)
    ws = S.workspace(S.saga_gather_workspace_size(g.plan, op, 32), device())
    torch.cuda.synchronize()
    sh = S.stream_handle(side)
    S.saga_scatter_apply_edge_gather(g.plan, op, inp, S.mat(out), C.c_void_p(ws.data_ptr()),
                                     ws.numel(), sh)
    S.saga_sync_check(sh)
    assert rel_err(to_np(out), O.gather(rp, col, X, "sum")) <= FP32_TOL


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_relabelling_moves_degrees_and_max_exactly(dtype):
    """Permutation equivariance where it is exact: the vertices of a
    power-law graph relabelled by a seeded permutation pi (in-CSR rebuilt,
    source rows moved with their labels).  The plan's in- and out-degrees
    move with the labels bit for bit, and so does the max Gather's output."""
    from synth import graphs as G

    S = lib()
    rp, col, n = _power_law()
    pi = G.rng_for(1603, 5).permutation(n)
    dst = np.repeat(np.arange(n), np.diff(rp))
    rp2, col2 = G.to_in_csr(n, pi[col], pi[dst])
    g1 = graph(rp, col, num_src=n, seg_len=16, block_cost=128, row_cost=4)
    g2 = graph(rp2, col2, num_src=n, seg_len=16, block_cost=128, row_cost=4)
    a1 = {k: v.cpu().numpy() for k, v in g1.arrays().items()}
    a2 = {k: v.cpu().numpy() for k, v in g2.arrays().items()}
    assert np.array_equal(a2["d_in"][pi], a1["d_in"])
    assert np.array_equal(a2["d_out"][pi], a1["d_out"])
    F = 64
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    X = np.random.default_rng(5).standard_normal((n, F)).astype(np.float32)
    if dtype == "bf16":
        X = _bf16_round(X)
    X2 = X[np.argsort(pi)]  # row pi[u] of X2 is row u of X
    print(f"relabelled max gather {dtype}", flush=True)
    o1 = to_np(run_gather(g1, dev_padded(X, tdt), dict(reduce=S.SAGA_RED_MAX), F, tdt))
    o2 = to_np(run_gather(g2, dev_padded(X2, tdt), dict(reduce=S.SAGA_RED_MAX), F, tdt))
    assert np.array_equal(o2[pi], o1)


@pytest.mark.parametrize("gname", ["rmat", "tiny_multi", "tiny_star"])
@pytest.mark.parametrize("heads,D", [(4, 8), (8, 8), (1, 4)])
def test_gather_attention_weights_sum_to_one(gname, heads, D):
    """Edge-softmax invariant (Sec. 3.2 attention scores normalised over a
    destination's in-edges): with every source row z_u = 1, each head's
    output is the sum of its attention weights, 1 for a non-empty row
    (within d_in * 2^-23 in float32) and 0 for an empty one.  The scores
    span about +-100, so the max subtraction and the merge of split rows
    (segments of 16 edges) are exercised."""
    S = lib()
    rp, col, n, g = _get_graph(gname)
    F = heads * D
    rng = np.random.default_rng(19 + heads)
    Zx = np.ones((n, F + 2 * heads), np.float32)
    Zx[:, F:] = (rng.standard_normal((n, 2 * heads)) * 30).astype(np.float32)
    zt = dev_padded(Zx, torch.float32)
    print(f"gather attention sum-to-one {gname} H={heads} D={D}", flush=True)
    out = run_gather(g, zt[:, :F], dict(msg=S.SAGA_MSG_GAT, reduce=S.SAGA_RED_SOFTMAX, heads=heads,
                                        neg_slope=0.2), F, torch.float32,
                     el=zt[:, F:F + heads], er=zt[:, F + heads:])
    got = to_np(out).astype(np.float64)
    d = np.diff(rp).astype(np.float64)
    want = np.broadcast_to((d > 0)[:, None], got.shape).astype(np.float64)
    assert np.all(np.abs(got - want) <= np.maximum(d, 1.0)[:, None] * 2.0**-23)


@pytest.mark.parametrize("gname", ["rmat", "tiny_multi", "tiny_random"])
def test_gather_attention_zero_scores_is_mean(gname):
    """With el = er = 0 every score is 0, each weight is 1 / d_in, and the
    attention Gather is the mean Gather of z (the oracle's mean, not its
    attention code, is the reference)."""
    S = lib()
    rp, col, n, g = _get_graph(gname)
    heads, D = 8, 8
    F = heads * D
    rng = np.random.default_rng(23)
    Zx = np.zeros((n, F + 2 * heads), np.float32)
    Zx[:, :F] = rng.standard_normal((n, F)).astype(np.float32)
    zt = dev_padded(Zx, torch.float32)
    print(f"gather attention zero scores {gname}", flush=True)
    out = run_gather(g, zt[:, :F], dict(msg=S.SAGA_MSG_GAT, reduce=S.SAGA_RED_SOFTMAX, heads=heads,
                                        neg_slope=0.2), F, torch.float32,
                     el=zt[:, F:F + heads], er=zt[:, F + heads:])
    assert rel_err(to_np(out), O.gather(rp, col, Zx[:, :F], "mean")) <= FP32_TOL


@pytest.mark.parametrize("gname", ["rmat", "tiny_multi", "tiny_chain"])
def test_gather_gated(gname):
    """Gated messages: the kernel gets the split form (gate_src = H W_src,
    gate_dst = H W_dst, W_edge); the oracle evaluates the concatenated
    definition [h_u | h_v | e_uv] W_e + b_e directly."""
    S = lib()
    rp, col, n, g = _get_graph(gname)
    E = len(col)
    F, Fe = 64, 16
    rng = np.random.default_rng(11)
    H = rng.standard_normal((n, F)).astype(np.float32)
    Ef = rng.standard_normal((E, Fe)).astype(np.float32)
    W_e = (rng.standard_normal((2 * F + Fe, F)) * 0.1).astype(np.float32)
    b_e = rng.standard_normal(F).astype(np.float32)
    Gs = (H.astype(np.float64) @ W_e[:F]).astype(np.float32)
    Gd = (H.astype(np.float64) @ W_e[F:2 * F]).astype(np.float32)
    t = lambda a: dev_padded(a, torch.float32)  # noqa: E731
    Ht, Gst, Gdt, Eft = t(H), t(Gs), t(Gd), t(Ef)
    wt = torch.from_numpy(W_e[2 * F:].copy()).to(device())
    bt = torch.from_numpy(b_e).to(device())
    extra = dict(gate_src=S.cmat(Gst), gate_dst=S.cmat(Gdt), edge_feat=S.cmat(Eft),
                 w_edge=wt.data_ptr(), gate_bias=bt.data_ptr())
    print(f"gather gated {gname}", flush=True)
    out = run_gather(g, Ht, dict(msg=S.SAGA_MSG_GATED, reduce=S.SAGA_RED_SUM), F, torch.float32,
                     extra=extra)
    ref = O.gated_gather(rp, col, H, Ef, W_e, b_e)
    assert rel_err(to_np(out), ref) <= FP32_TOL


@pytest.fixture(scope="module")
def blocky():
    """R-MAT with 2^16 vertices and 1 M edges, planned with 256-cost row
    blocks and 64-edge segments: about 5,400 blocks, so the launcher hands
    each workgroup four consecutive blocks (blocks are paired up while a
    workgroup holds at most 2048 cost units and 1024 workgroups remain)."""
    from synth import configs as C_

    d = C_.build("sage_rmat", scale=16, key=1603)
    rp, col, n = d["row_ptr"], d["col_idx"], d["num_vertices"]
    return rp, col, n, graph(rp, col, num_src=n, seg_len=64, block_cost=256, row_cost=4)


@pytest.mark.parametrize("F", [64, 256])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gather_merged_blocks(blocky, F, dtype):
    S = lib()
    rp, col, n, g = blocky
    rng = np.random.default_rng(F + 1)
    X = rng.standard_normal((n, F)).astype(np.float32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    if dtype == "bf16":
        X = _bf16_round(X)
    Xt = dev_padded(X, tdt)
    tol = FP32_TOL if dtype == "f32" else BF16_TOL
    bias = rng.standard_normal(F)
    for red, msg, dn, b, act in [("sum", "copy", 0, None, "none"),
                                 ("mean", "src_norm", 1, bias, "relu")]:
        print(f"gather merged blocks F={F} {dtype} {red} {msg}", flush=True)
        out = run_gather(g, Xt, dict(reduce={"sum": S.SAGA_RED_SUM, "mean": S.SAGA_RED_MEAN}[red],
                                     msg={"copy": S.SAGA_MSG_COPY, "src_norm": S.SAGA_MSG_SRC_NORM}[msg],
                                     dst_norm=dn, act=act), F, tdt, bias=b)
        assert rel_err(to_np(out), _ref_simple(rp, col, X, red, msg, dn, b, act, n)) <= tol
    print(f"gather merged blocks F={F} {dtype} max", flush=True)
    out = run_gather(g, Xt, dict(reduce=S.SAGA_RED_MAX), F, tdt)
    assert np.array_equal(to_np(out), O.gather(rp, col, X, "max"))


def test_gather_attention_and_gated_merged_blocks(blocky):
    S = lib()
    rp, col, n, g = blocky
    rng = np.random.default_rng(3)
    heads, D = 8, 8
    F = heads * D
    Zx = rng.standard_normal((n, F + 2 * heads)).astype(np.float32)
    zt = dev_padded(Zx, torch.float32)
    print("gather attention merged blocks", flush=True)
    out = run_gather(g, zt[:, :F], dict(msg=S.SAGA_MSG_GAT, reduce=S.SAGA_RED_SOFTMAX, heads=heads,
                                        neg_slope=0.2), F, torch.float32,
                     el=zt[:, F:F + heads], er=zt[:, F + heads:])
    ref = O.attention_gather(rp, col, Zx[:, :F], Zx[:, F:F + heads], Zx[:, F + heads:], heads, 0.2)
    assert rel_err(to_np(out), ref) <= FP32_TOL
    E = len(col)
    Fe = 16
    H = rng.standard_normal((n, F)).astype(np.float32)
    Ef = rng.standard_normal((E, Fe)).astype(np.float32)
    W_e = (rng.standard_normal((2 * F + Fe, F)) * 0.1).astype(np.float32)
    b_e = rng.standard_normal(F).astype(np.float32)
    Gs = (H.astype(np.float64) @ W_e[:F]).astype(np.float32)
    Gd = (H.astype(np.float64) @ W_e[F:2 * F]).astype(np.float32)
    t = lambda a: dev_padded(a, torch.float32)  # noqa: E731
    Ht, Gst, Gdt, Eft = t(H), t(Gs), t(Gd), t(Ef)
    wt = torch.from_numpy(W_e[2 * F:].copy()).to(device())
    bt = torch.from_numpy(b_e).to(device())
    extra = dict(gate_src=S.cmat(Gst), gate_dst=S.cmat(Gdt), edge_feat=S.cmat(Eft),
                 w_edge=wt.data_ptr(), gate_bias=bt.data_ptr())
    print("gather gated merged blocks", flush=True)
    out = run_gather(g, Ht, dict(msg=S.SAGA_MSG_GATED, reduce=S.SAGA_RED_SUM), F, torch.float32,
                     extra=extra)
    assert rel_err(to_np(out), O.gated_gather(rp, col, H, Ef, W_e, b_e)) <= FP32_TOL


def test_gather_deterministic():
    S = lib()
    rp, col, n, g = _get_graph("rmat")
    X = np.random.default_rng(5).standard_normal((n, 128)).astype(np.float32)
    Xt = dev_padded(X)
    a = run_gather(g, Xt, dict(reduce=S.SAGA_RED_SUM, dst_norm=1), 128, torch.float32)
    b = run_gather(g, Xt, dict(reduce=S.SAGA_RED_SUM, dst_norm=1), 128, torch.float32)
    assert torch.equal(a.cpu(), b.cpu())


# --------------------------------------------------------------------------
# ApplyVertex GEMM
# --------------------------------------------------------------------------
def run_gemm(A, W, dtype, bias=None, act="none", deg=None, A2=None, W2=None, bias2=None,
             mode="plain", out_cols=None):
    S = lib()
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    op = S.saga_gemm_op()
    op.dtype = S.dtype_code(tdt)
    op.mode = {"plain": 0, "concat": 1, "gru": 2}[mode]
    op.act = ACTS[act]
    dev = device()
    keep = []
    if deg is not None:
        dt = torch.from_numpy(np.asarray(deg, np.int32)).to(dev)
        keep.append(dt)
        op.row_scale_deg = dt.data_ptr()
    At = dev_padded(A, tdt)
    Wt = torch.from_numpy(np.asarray(W, np.float32)).to(tdt).to(dev)
    A2t = dev_padded(A2, tdt) if A2 is not None else None
    W2t = torch.from_numpy(np.asarray(W2, np.float32)).to(tdt).to(dev) if W2 is not None else None
    bt = torch.from_numpy(np.asarray(bias, np.float32)).to(dev) if bias is not None else None
    b2t = torch.from_numpy(np.asarray(bias2, np.float32)).to(dev) if bias2 is not None else None
    M = A.shape[0]
    N = out_cols or W.shape[1]
    out = dev_padded(np.zeros((M, N)), tdt, fill=3.0)
    nws = S.saga_apply_vertex_workspace_size(op, A.shape[1], 0 if A2 is None else A2.shape[1],
                                             W.shape[1])
    ws = S.workspace(nws, dev)
    S.saga_apply_vertex(op, S.cmat(At), S.cmat(Wt), S.cmat(A2t), S.cmat(W2t),
                        None if bt is None else bt.data_ptr(),
                        None if b2t is None else b2t.data_ptr(), S.mat(out),
                        C.c_void_p(ws.data_ptr()), ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("M,K,N", [(1000, 602, 128), (777, 128, 41), (2000, 128, 16),
                                   (130, 16, 8), (513, 512, 80), (300, 256, 256),
                                   (64, 64, 192), (5, 37, 3)])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gemm_plain(M, K, N, dtype):
    rng = np.random.default_rng(M + K + N)
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    if dtype == "bf16":
        A, W = _bf16_round(A), _bf16_round(W)
    bias = rng.standard_normal(N)
    deg = rng.integers(0, 9, M)
    print(f"gemm plain M={M} K={K} N={N} {dtype}", flush=True)
    out = run_gemm(A, W, dtype, bias=bias, act="relu", deg=deg)
    ref = O.dense(A, W, bias=bias, act="relu", row_scale=O.degree_scale(deg))
    assert rel_err(to_np(out), ref) <= (FP32_TOL if dtype == "f32" else BF16_TOL)
    out = run_gemm(A, W, dtype)
    ref = O.dense(A, W)
    assert rel_err(to_np(out), ref) <= (FP32_TOL if dtype == "f32" else BF16_TOL)


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gemm_plain_many_tiles(dtype):
    """More 128-row tiles than the device holds workgroups at once (later
    waves of workgroups reuse the LDS of earlier ones), a ragged last tile
    and a K tail, with the row scale, bias and activation epilogue."""
    rng = np.random.default_rng(9)
    M, K, N = 200_003, 150, 128
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    if dtype == "bf16":
        A, W = _bf16_round(A), _bf16_round(W)
    bias = rng.standard_normal(N)
    deg = rng.integers(0, 9, M)
    print(f"gemm plain many tiles M={M} K={K} N={N} {dtype}", flush=True)
    out = run_gemm(A, W, dtype, bias=bias, act="relu", deg=deg)
    ref = O.dense(A, W, bias=bias, act="relu", row_scale=O.degree_scale(deg))
    assert rel_err(to_np(out), ref) <= (FP32_TOL if dtype == "f32" else BF16_TOL)


@pytest.mark.parametrize("M,K,N,act", [(4099, 602, 128, "relu"), (1000, 608, 100, "elu"),
                                       (3001, 300, 81, "none"), (2050, 256, 128, "tanh"),
                                       (17, 512, 96, "sigmoid"), (100_003, 602, 128, "relu"),
                                       (5000, 192, 128, "relu"), (33, 255, 90, "elu")])
def test_gemm_bf16_resident_weights(M, K, N, act):
    """bfloat16 products with 80 < N <= 128 and 192 <= K <= 608 (the
    weights held in LDS for the whole run, rows streamed per wave, stores
    through lane exchanges): ragged M, K and N, fewer rows than one wave's
    tile, and more tiles than waves, with the full epilogue."""
    rng = np.random.default_rng(M + K + N)
    A = _bf16_round(rng.standard_normal((M, K)).astype(np.float32))
    W = _bf16_round((rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32))
    bias = rng.standard_normal(N)
    deg = rng.integers(0, 9, M)
    print(f"gemm bf16 resident M={M} K={K} N={N} {act}", flush=True)
    out = run_gemm(A, W, "bf16", bias=bias, act=act, deg=deg)
    ref = O.dense(A, W, bias=bias, act=act, row_scale=O.degree_scale(deg))
    assert rel_err(to_np(out), ref) <= BF16_TOL
    out = run_gemm(A, W, "bf16")
    assert rel_err(to_np(out), O.dense(A, W)) <= BF16_TOL


def test_gemm_small_integers_exact():
    rng = np.random.default_rng(1)
    A = rng.integers(-8, 9, (333, 64)).astype(np.float32)
    W = rng.integers(-8, 9, (64, 48)).astype(np.float32)
    exact = A.astype(np.float64) @ W
    out = run_gemm(A, W, "f32")
    assert np.array_equal(to_np(out), exact)
    # bf16 storage: products and sums are exact in the fp32 accumulator, the
    # stored result is the round-to-nearest-even bf16 of the exact integer
    out = run_gemm(A, W, "bf16")
    assert np.array_equal(to_np(out), _bf16_round(exact))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_gemm_concat(dtype):
    rng = np.random.default_rng(2)
    M, K1, K2, N = 700, 256, 200, 256
    A = rng.standard_normal((M, K1)).astype(np.float32)
    A2 = rng.standard_normal((M, K2)).astype(np.float32)
    W = (rng.standard_normal((K1, N)) / 16).astype(np.float32)
    W2 = (rng.standard_normal((K2, N)) / 16).astype(np.float32)
    if dtype == "bf16":
        A, A2, W, W2 = map(_bf16_round, (A, A2, W, W2))
    b = rng.standard_normal(N)
    out = run_gemm(A, W, dtype, bias=b, A2=A2, W2=W2, mode="concat")
    ref = O.dense(np.concatenate([A, A2], 1), np.concatenate([W, W2], 0), bias=b)
    assert rel_err(to_np(out), ref) <= (FP32_TOL if dtype == "f32" else BF16_TOL)


@pytest.mark.parametrize("F", [16, 64])
def test_gemm_gru(F):
    rng = np.random.default_rng(F)
    M = 1001
    a = rng.standard_normal((M, F)).astype(np.float32)
    h = rng.standard_normal((M, F)).astype(np.float32)
    Wih = (rng.standard_normal((F, 3 * F)) / 8).astype(np.float32)
    Whh = (rng.standard_normal((F, 3 * F)) / 8).astype(np.float32)
    bih = rng.standard_normal(3 * F)
    bhh = rng.standard_normal(3 * F)
    out = run_gemm(a, Wih, "f32", bias=bih, A2=h, W2=Whh, bias2=bhh, mode="gru", out_cols=F)
    ref = O.gru_cell(a, h, Wih, bih, Whh, bhh)
    assert rel_err(to_np(out), ref) <= FP32_TOL


@pytest.mark.parametrize("dtype,N,split,K,aligned", [
    ("f32", 41, 32, 150, False), ("f32", 100, 64, 150, False), ("bf16", 100, 64, 150, False),
    ("bf16", 128, 64, 602, False), ("bf16", 100, 41, 300, False), ("bf16", 128, 64, 602, True),
    ("bf16", 100, 41, 300, True), ("f32", 100, 64, 150, True)])
def test_gemm_split_output_equals_single_output(dtype, N, split, K, aligned):
    """split_col writes columns [0, s) to out and [s, N) to the tail matrix:
    the same values, bit for bit, as one output matrix (row scale, bias and
    activation included)."""
    S = lib()
    rng = np.random.default_rng(N)
    M = 777
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = rng.standard_normal((K, N)).astype(np.float32) / np.sqrt(K)
    b = rng.standard_normal(N).astype(np.float32)
    deg = torch.from_numpy(rng.integers(0, 9, M).astype(np.int32)).to(device())
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    a = dev_padded(A, dtype=tdt)
    w = torch.from_numpy(W).to(device()).to(tdt)
    bias = torch.from_numpy(b).to(device())
    op = S.saga_gemm_op(S.dtype_code(tdt), S.SAGA_GEMM_PLAIN, S.SAGA_ACT_ELU, deg.data_ptr())
    ws = S.workspace(S.saga_apply_vertex_workspace_size(op, K, 0, N), device())
    none = S.saga_cmat(None, 0, 0, 0)
    print(f"gemm split {dtype} N={N} s={split} K={K} aligned={aligned}", flush=True)
    one = torch.full((M, N), 7.0, dtype=tdt, device=device())
    S.saga_apply_vertex(op, S.cmat(a), S.cmat(w), none, none, bias.data_ptr(), None, S.mat(one),
                        C.c_void_p(ws.data_ptr()), ws.numel(), S.stream_handle())
    # head and tail rows padded to 16 bytes (whole-piece stores) or the tail
    # by 3 elements (element stores)
    per16 = 16 // (4 if dtype == "f32" else 2)
    ld_head = -(-split // per16) * per16 if aligned else split
    ld_tail = -(-(N - split) // per16) * per16 if aligned else N - split + 3
    head = torch.full((M, ld_head), 7.0, dtype=tdt, device=device())[:, :split]
    tail = torch.full((M, ld_tail), 7.0, dtype=tdt, device=device())[:, :N - split]
    op.split_col = split
    op.tail = S.mat(tail)
    S.saga_apply_vertex(op, S.cmat(a), S.cmat(w), none, none, bias.data_ptr(), None, S.mat(head),
                        C.c_void_p(ws.data_ptr()), ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    assert torch.equal(head, one[:, :split]) and torch.equal(tail, one[:, split:])
    op.split_col = N  # must be inside (0, N)
    with pytest.raises(S.SagaError):
        S.saga_apply_vertex(op, S.cmat(a), S.cmat(w), none, none, None, None, S.mat(head),
                            C.c_void_p(ws.data_ptr()), ws.numel(), S.stream_handle())


@pytest.mark.parametrize("dtype,F", [("f32", 512), ("bf16", 1024), ("f32", 508), ("bf16", 1000),
                                     ("f32", 602), ("f32", 1024), ("f32", 1000), ("bf16", 602)])
def test_gather_maximum_widths(dtype, F):
    """Wide rows up to the widest the simple Gather takes (1024 columns in
    both dtypes; float32 rows past 512 columns run as 128-byte slices, 602
    and 1000 with a ragged last slice), sum with both norms and max, on the
    power-law graph with split rows."""
    S = lib()
    rp, col, n, g = _get_graph("rmat")
    rng = np.random.default_rng(F)
    X = rng.standard_normal((n, F)).astype(np.float32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    if dtype == "bf16":
        X = _bf16_round(X)
    Xt = dev_padded(X, tdt)
    tol = FP32_TOL if dtype == "f32" else BF16_TOL
    print(f"gather max width {dtype} F={F}", flush=True)
    out = run_gather(g, Xt, dict(reduce=S.SAGA_RED_SUM, msg=S.SAGA_MSG_SRC_NORM, dst_norm=1,
                                 act="none"), F, tdt)
    ref = _ref_simple(rp, col, X, "sum", "src_norm", 1, None, "none", n)
    assert rel_err(to_np(out), ref) <= tol
    out = run_gather(g, Xt, dict(reduce=S.SAGA_RED_MAX), F, tdt)
    assert np.array_equal(to_np(out), O.gather(rp, col, X, "max"))
    limit = 1024  # one column past the widest row is refused
    wider = dev_padded(np.zeros((n, limit + 1), np.float32), tdt)
    with pytest.raises(S.SagaError):
        run_gather(g, wider, dict(reduce=S.SAGA_RED_SUM), limit + 1, tdt)


def _transform_ref(rp, col, X, red, dn, bias, act, nsrc, W, rs_deg, dtype="f32"):
    """out[v] = rs(v) * (h_v W) with h the Gather output (the fused call's
    definition), from the oracle's Gather and a float64 product.  In bf16, h
    is a stored intermediate of the call, so it is taken rounded to bf16
    (the bf16 contract: storage in bf16, arithmetic in float64 here)."""
    h = _ref_simple(rp, col, X, red, "copy", dn, bias, act, nsrc)
    if dtype == "bf16":
        h = _bf16_round(h.astype(np.float32)).astype(np.float64)
    rs = O.degree_scale(rs_deg) if rs_deg is not None else np.ones(h.shape[0])
    return O.dense(h, W) * rs[:, None], h


@pytest.mark.parametrize("gname", ["rmat", "tiny_multi", "tiny_random", "edgeless"])
@pytest.mark.parametrize("dtype,F,N,split", [("f32", 128, 41, 32), ("f32", 32, 8, 0), ("f32", 64, 64, 0),
                                             ("bf16", 128, 41, 0), ("bf16", 64, 16, 8)])
def test_gather_transform_fused(gname, dtype, F, N, split):
    """The Gather with the next layer's transform fused into its last slice
    pass: against the oracle's definition (Gather, then the product with the
    row scale), and against the two separate calls it replaces."""
    S = lib()
    rp, col, n, g = _get_graph(gname)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    rng = np.random.default_rng(60 + F + N)
    X = rng.standard_normal((n, F)).astype(np.float32)
    W = (rng.standard_normal((F, N)) / np.sqrt(F)).astype(np.float32)
    if dtype == "bf16":
        X, W = _bf16_round(X), _bf16_round(W)
    bias = rng.standard_normal(F)
    tol = FP32_TOL if dtype == "f32" else BF16_TOL
    d_out = O.out_degrees(col, n)
    dout_t = torch.from_numpy(d_out.astype(np.int32)).to(device())
    Xt, Wt = dev_padded(X, tdt), torch.from_numpy(W).to(tdt).to(device()).contiguous()
    b_t = torch.from_numpy(bias.astype(np.float32)).to(device())
    for red, dn, act, rsd in (("sum", 1, "relu", d_out), ("mean", 0, "none", None)):
        print(f"gather+transform {gname} {dtype} F={F} N={N} split={split} {red}", flush=True)
        op = S.saga_edge_op(S.SAGA_MSG_COPY, {"sum": S.SAGA_RED_SUM, "mean": S.SAGA_RED_MEAN}[red],
                            S.dtype_code(tdt), 1, 0, dn, 0.0, ACTS[act])
        inp = S.saga_edge_inputs()
        inp.src = S.cmat(Xt)
        inp.bias = b_t.data_ptr()
        head = split if split else N
        out = dev_padded(np.zeros((n, head)), dtype=tdt, fill=7.0)
        tail = dev_padded(np.zeros((n, N - split)), dtype=tdt, fill=7.0) if split else None
        nx = S.saga_next_transform()
        nx.w = S.cmat(Wt)
        nx.row_scale_deg = dout_t.data_ptr() if rsd is not None else None
        nx.split_col = split
        if split:
            nx.tail = S.mat(tail)
        ws = S.workspace(S.saga_gather_transform_workspace_size(g.plan, op, F), device())
        S.saga_scatter_apply_edge_gather_transform(g.plan, op, inp, nx, S.mat(out),
                                                   C.c_void_p(ws.data_ptr()), ws.numel(), S.stream_handle())
        torch.cuda.synchronize()
        got = to_np(out) if not split else np.concatenate([to_np(out), to_np(tail)], axis=1)
        ref, h = _transform_ref(rp, col, X, red, dn, bias, act, n, W, rsd, dtype)
        mag = O.dense(np.abs(h), np.abs(W)) * (O.degree_scale(rsd)[:, None] if rsd is not None else 1.0)
        assert rel_err(got, ref) <= tol
        assert rel_err_terms(got, ref, mag) <= tol
        # the two calls it replaces: Gather, then the transform on the stored h
        hh = run_gather(g, Xt, dict(reduce=op.reduce, dst_norm=dn, act=act), F, tdt, bias=bias)
        gop = S.saga_gemm_op(S.dtype_code(tdt), S.SAGA_GEMM_PLAIN, S.SAGA_ACT_NONE,
                             dout_t.data_ptr() if rsd is not None else None)
        y2 = dev_padded(np.zeros((n, N)), dtype=tdt)
        gws = S.workspace(S.saga_apply_vertex_workspace_size(gop, F, 0, N), device())
        none = S.saga_cmat(None, 0, 0, 0)
        S.saga_apply_vertex(gop, S.cmat(hh), S.cmat(Wt), none, none, None, None, S.mat(y2),
                            C.c_void_p(gws.data_ptr()), gws.numel(), S.stream_handle())
        torch.cuda.synchronize()
        assert rel_err(got, to_np(y2)) <= tol
