"""Seeded sweeps over the corners of the layout, the Gather and the GEMM.

Layout and Gather: random
graphs (empty-heavy, uniform, power-law, one giant row; fewer or more
source vertices than destinations), random plan options (segment lengths
from 1, row costs, block costs down to the smallest allowed, which also
makes the launcher hand several blocks to a workgroup), random widths
(1 to 129 columns, fp32 and bf16) and every simple reduction.  The plan is
compared with the oracle's bit for bit, the Gathers element by element.
GEMM: random shapes over every tile path and epilogue, and a sweep over
the shapes the bfloat16 weight-resident kernel takes."""
import numpy as np
import pytest
import torch

from gpu_util import dev_padded, graph, lib, to_np
from helpers import BF16_TOL, FP32_TOL, rel_err
from oracle import saga_oracle as O

pytestmark = pytest.mark.gpu

CASES = 200


def _bf16_round(a):
    from synth import tensors as T

    return T.bf16_to_f32(T.bf16_bits(np.asarray(a, np.float32)))


def _random_graph(rng):
    V = int(rng.integers(1, 3000))
    Vs = int(rng.choice([V, max(1, V // 3), V + int(rng.integers(1, 500))]))
    kind = rng.choice(["empty", "uniform", "power", "giant"])
    if kind == "empty":
        d = np.where(rng.random(V) < 0.8, 0, rng.integers(1, 20, V))
    elif kind == "uniform":
        d = rng.integers(0, 12, V)
    elif kind == "power":
        d = np.minimum(rng.zipf(1.6, V) - 1, 5000)
    else:
        d = rng.integers(0, 4, V)
        d[int(rng.integers(0, V))] = int(rng.integers(2000, 20000))
    rp = np.zeros(V + 1, np.int64)
    np.cumsum(d, out=rp[1:])
    col = rng.integers(0, Vs, int(rp[-1])).astype(np.int32)
    # CSR order within a row: by source id (ties keep order)
    for v in np.flatnonzero(d > 1):
        col[rp[v]:rp[v + 1]] = np.sort(col[rp[v]:rp[v + 1]], kind="stable")
    return rp.astype(np.int32), col, V, Vs, kind


@pytest.mark.parametrize("case", range(CASES))
def test_fuzz_plan_and_gather(case):
    S = lib()
    rng = np.random.default_rng(9000 + case)
    rp, col, V, Vs, kind = _random_graph(rng)
    T = int(rng.choice([1, 2, 3, 5, 8, 16, 33, 64, 512]))
    c = int(rng.integers(1, 9))
    B = T + c + int(rng.choice([0, 1, 7, 100, 1000]))
    F = int(rng.choice([1, 2, 3, 4, 5, 8, 17, 32, 33, 64, 100, 128, 129]))
    dtype = str(rng.choice(["f32", "bf16"]))
    print(f"fuzz case {case}: {kind} V={V} Vs={Vs} E={len(col)} seg_len={T} row_cost={c} "
          f"block_cost={B} F={F} {dtype}", flush=True)
    g = graph(rp, col, num_src=Vs, seg_len=T, block_cost=B, row_cost=c)
    got = {k: v.cpu().numpy().astype(np.int64) for k, v in g.arrays().items()}
    want = O.plan(rp, col, Vs, T, B, c)
    for k in ("d_in", "d_out", "perm", "row_seg_first", "seg_row", "seg_beg", "seg_end",
              "block_ptr"):
        assert np.array_equal(got[k], want[k]), k
    assert g.counts.n_split == want["n_split"]

    X = rng.standard_normal((Vs, F)).astype(np.float32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    if dtype == "bf16":
        X = _bf16_round(X)
    Xt = dev_padded(X, tdt)
    tol = FP32_TOL if dtype == "f32" else BF16_TOL
    from test_gpu_ops import run_gather

    for red in ("sum", "mean", "max"):
        code = {"sum": S.SAGA_RED_SUM, "mean": S.SAGA_RED_MEAN, "max": S.SAGA_RED_MAX}[red]
        out = to_np(run_gather(g, Xt, dict(reduce=code), F, tdt))
        ref = O.gather(rp, col, X, red)
        if red == "max":
            assert np.array_equal(out, ref), red
        else:
            assert rel_err(out, ref) <= tol, red


GEMM_CASES = 120


@pytest.mark.parametrize("case", range(GEMM_CASES))
def test_fuzz_gemm(case):
    """Random shapes across every tile path (narrow two- and four-stage
    tiles, the LDS-ring and register-A wide tiles, concat), ragged M, K and
    N, with a random epilogue (row scale, bias, activation)."""
    from test_gpu_ops import run_gemm

    rng = np.random.default_rng(7000 + case)
    M = int(rng.integers(1, 3000))
    K = int(rng.choice([1, 3, 16, 31, 32, 33, 64, 100, 128, 129, 255, 602, 700]))
    N = int(rng.choice([1, 3, 8, 16, 17, 41, 64, 80, 81, 96, 128, 129, 200, 256, 300]))
    dtype = str(rng.choice(["f32", "bf16"]))
    act = str(rng.choice(["none", "relu", "elu", "sigmoid", "tanh"]))
    concat = bool(rng.random() < 0.25)
    A = rng.standard_normal((M, K)).astype(np.float32)
    W = (rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32)
    A2 = W2 = None
    if concat:
        K2 = int(rng.choice([1, 32, 77, 128]))
        A2 = rng.standard_normal((M, K2)).astype(np.float32)
        W2 = (rng.standard_normal((K2, N)) / np.sqrt(K2)).astype(np.float32)
    if dtype == "bf16":
        A, W = _bf16_round(A), _bf16_round(W)
        if concat:
            A2, W2 = _bf16_round(A2), _bf16_round(W2)
    bias = rng.standard_normal(N) if rng.random() < 0.5 else None
    deg = rng.integers(0, 9, M) if rng.random() < 0.5 else None
    print(f"fuzz gemm {case}: M={M} K={K} N={N} {dtype} {act} concat={concat} "
          f"bias={bias is not None} deg={deg is not None}", flush=True)
    out = run_gemm(A, W, dtype, bias=bias, act=act, deg=deg, A2=A2, W2=W2,
                   mode="concat" if concat else "plain")
    AA = np.concatenate([A, A2], 1) if concat else A
    WW = np.concatenate([W, W2], 0) if concat else W
    ref = O.dense(AA, WW, bias=bias, act=act,
                  row_scale=None if deg is None else O.degree_scale(deg))
    assert rel_err(to_np(out), ref) <= (FP32_TOL if dtype == "f32" else BF16_TOL)


RESIDENT_CASES = 24


@pytest.mark.parametrize("case", range(RESIDENT_CASES))
def test_fuzz_gemm_bf16_resident(case):
    """bfloat16 PLAIN shapes the weight-resident kernel takes (80 < N <= 128,
    192 <= K <= 608): random M from one row to several tiles per wave,
    ragged K and N, random epilogue."""
    from test_gpu_ops import run_gemm

    rng = np.random.default_rng(9100 + case)
    M = int(rng.choice([1, 15, 16, 17, int(rng.integers(18, 5000)), int(rng.integers(30000, 70000))]))
    K = int(rng.integers(192, 609))
    N = int(rng.integers(81, 129))
    act = str(rng.choice(["none", "relu", "elu", "sigmoid", "tanh"]))
    A = _bf16_round(rng.standard_normal((M, K)).astype(np.float32))
    W = _bf16_round((rng.standard_normal((K, N)) / np.sqrt(K)).astype(np.float32))
    bias = rng.standard_normal(N) if rng.random() < 0.5 else None
    deg = rng.integers(0, 9, M) if rng.random() < 0.5 else None
    print(f"fuzz gemm resident {case}: M={M} K={K} N={N} {act} bias={bias is not None} "
          f"deg={deg is not None}", flush=True)
    out = run_gemm(A, W, "bf16", bias=bias, act=act, deg=deg)
    ref = O.dense(A, W, bias=bias, act=act, row_scale=None if deg is None else O.degree_scale(deg))
    assert rel_err(to_np(out), ref) <= BF16_TOL


def _small_graph(rng, vmax, dmax, long_row=0):
    V = int(rng.integers(1, vmax))
    d = rng.integers(0, dmax, V)
    d[rng.random(V) < 0.2] = 0
    if long_row and V > 1:
        d[int(rng.integers(0, V))] = long_row
    rp = np.zeros(V + 1, np.int64)
    np.cumsum(d, out=rp[1:])
    col = rng.integers(0, V, int(rp[-1])).astype(np.int32)
    for v in np.flatnonzero(d > 1):
        col[rp[v]:rp[v + 1]] = np.sort(col[rp[v]:rp[v + 1]], kind="stable")
    return rp.astype(np.int32), col, V


@pytest.mark.parametrize("case", range(40))
def test_fuzz_out_degrees(case):
    """The plan over graphs with many sources (log-uniform up to 2^23) and
    up to ~2e5 edges: several edge tiles with a ragged last one, hub
    sources, the first and last ids and ids on both sides of powers of
    two; d_out (and the rest of the plan) bit-exact against the oracle."""
    rng = np.random.default_rng(7000 + case)
    Vs = int(np.exp(rng.uniform(0.0, np.log(1 << 23))))
    V = int(rng.integers(1, 2000))
    d = rng.integers(0, int(rng.choice([2, 30, 200])), V)
    if rng.random() < 0.5:
        d[int(rng.integers(0, V))] = int(rng.integers(1000, 60000))
    rp = np.zeros(V + 1, np.int64)
    np.cumsum(d, out=rp[1:])
    E = int(rp[-1])
    col = rng.integers(0, Vs, E)
    if E:
        marks = [0, Vs - 1] + [x for k in range(1, 24) for x in ((1 << k) - 1, 1 << k)
                               if x < Vs]
        col[rng.integers(0, E, min(E, 4 * len(marks)))] = rng.choice(marks, min(E, 4 * len(marks)))
        hubs = rng.integers(0, Vs, int(rng.integers(1, 6)))
        k = int(rng.integers(0, E // 2 + 1))
        col[rng.integers(0, E, k)] = rng.choice(hubs, k)
    T = int(rng.choice([4, 64, 512]))
    c = int(rng.integers(1, 9))
    print(f"fuzz out-degrees {case}: V={V} Vs={Vs} E={E} seg_len={T} row_cost={c}", flush=True)
    g = graph(rp.astype(np.int32), col.astype(np.int32), num_src=Vs, seg_len=T,
              block_cost=T + c + 100, row_cost=c)
    got = {k: v.cpu().numpy().astype(np.int64) for k, v in g.arrays().items()}
    want = O.plan(rp, col, Vs, T, T + c + 100, c)
    for k in ("d_in", "d_out", "perm", "row_seg_first", "seg_row", "seg_beg", "seg_end",
              "block_ptr"):
        assert np.array_equal(got[k], want[k]), k
    assert g.counts.error_flags == 0


@pytest.mark.parametrize("case", range(60))
def test_fuzz_attention(case):
    """Edge-softmax Gather over random graphs, head counts and widths."""
    from test_gpu_ops import run_gather

    S = lib()
    rng = np.random.default_rng(5000 + case)
    rp, col, V, Vs, kind = _random_graph(rng)
    H = int(rng.choice([1, 2, 4, 8, 16]))
    D = int(rng.choice([d for d in (4, 8, 12, 16, 32, 64) if H * d <= 256]))
    F = H * D
    head_mean = int(rng.random() < 0.4 and (F // 4) & (F // 4 - 1) == 0)
    T = int(rng.choice([1, 4, 16, 64, 512]))
    c = int(rng.integers(1, 9))
    g = graph(rp, col, num_src=Vs, seg_len=T, block_cost=T + c + int(rng.choice([0, 50, 900])),
              row_cost=c)
    Z = rng.standard_normal((Vs, F + H)).astype(np.float32)
    er = rng.standard_normal((V, H)).astype(np.float32)
    zt, ert = dev_padded(Z), dev_padded(er)
    bias = rng.standard_normal(D if head_mean else F)
    print(f"fuzz attention {case}: {kind} V={V} Vs={Vs} E={len(col)} H={H} D={D} "
          f"mean={head_mean} seg_len={T}", flush=True)
    out = run_gather(g, zt[:, :F], dict(msg=S.SAGA_MSG_GAT, reduce=S.SAGA_RED_SOFTMAX, heads=H,
                                        head_mean=head_mean, act="elu", neg_slope=0.2),
                     D if head_mean else F, torch.float32, el=zt[:, F:], er=ert, bias=bias)
    o = O.attention_gather(rp, col, Z[:, :F], Z[:, F:], er, H, 0.2)
    if head_mean:
        o = o.reshape(V, H, D).mean(axis=1)
    assert rel_err(to_np(out), O.elu(o + bias[None, :])) <= FP32_TOL


@pytest.mark.parametrize("case", range(40))
def test_fuzz_rgcn_layer(case):
    """R-GCN layers over random graphs, relation counts, type skews and
    widths (typed layout, grouped transform, typed Gather with self term)."""
    from paper_2009_00804_amd import layers as LY

    S = lib()
    rng = np.random.default_rng(6000 + case)
    rp, col, V = _small_graph(rng, 1200, int(rng.choice([3, 12, 40])),
                              long_row=int(rng.choice([0, 0, 2500])))
    R = int(rng.choice([1, 2, 3, 7, 32]))
    p = 1.0 / (np.arange(R) + 1.0) ** float(rng.choice([0.0, 1.0, 2.0]))
    et = rng.choice(R, size=len(col), p=p / p.sum()).astype(np.int32)
    Fi = int(rng.choice([4, 20, 64, 128]))
    Fo = int(rng.choice([8, 36, 64, 100]))
    dtype = str(rng.choice(["f32", "bf16"]))
    X = rng.standard_normal((V, Fi)).astype(np.float32)
    W_rel = (rng.standard_normal((R, Fi, Fo)) / np.sqrt(Fi)).astype(np.float32)
    W_self = (rng.standard_normal((Fi, Fo)) / np.sqrt(Fi)).astype(np.float32)
    b = (rng.standard_normal(Fo) * 0.1).astype(np.float32)
    if dtype == "bf16":
        X, W_rel, W_self = _bf16_round(X), _bf16_round(W_rel), _bf16_round(W_self)
    print(f"fuzz rgcn {case}: V={V} E={len(col)} R={R} {Fi}->{Fo} {dtype}", flush=True)
    g = graph(rp, col)
    rg = S.RelGraph(g, torch.from_numpy(et).to(g.row_ptr.device), R)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    model = LY.rgcn(g, rg, dict(W_rel=W_rel, W_self=W_self, b=b, act="relu"), dtype=tdt)
    y = LY.run(model, dev_padded(X, dtype=tdt))
    torch.cuda.synchronize()
    want = O.rgcn_layer(rp, col, et, X, W_rel, W_self, b, act="relu")
    assert rel_err(to_np(y), want) <= (FP32_TOL if dtype == "f32" else BF16_TOL)


@pytest.mark.parametrize("case", range(24))
def test_fuzz_lstm_gather(case):
    """LSTM Gather over random graphs (empty rows, a long row) and H."""
    from test_gpu_lstm import _ref, run_lstm

    rng = np.random.default_rng(4000 + case)
    rp, col, V = _small_graph(rng, 400, int(rng.choice([2, 10, 60])),
                              long_row=int(rng.choice([0, 1100, 2100])))
    H = int(rng.choice([32, 64, 128]))
    P = (rng.standard_normal((V, 4 * H)) * 0.5).astype(np.float32)
    W_hh = (rng.standard_normal((H, 4 * H)) / np.sqrt(H)).astype(np.float32)
    print(f"fuzz lstm {case}: V={V} E={len(col)} H={H}", flush=True)
    g = graph(rp, col)
    assert rel_err(run_lstm(g, P, W_hh), _ref(rp, col, P, W_hh)) <= FP32_TOL


@pytest.mark.parametrize("case", range(24))
def test_fuzz_gated_and_unfused(case):
    """Gated-message Gather (edge features of 4 to 16 columns) and the
    unfused baseline (edge tensor, then segment reduction) over random
    graphs and plan options."""
    from test_gpu_ops import run_gather
    from test_gpu_unfused import run_unfused

    S = lib()
    rng = np.random.default_rng(3000 + case)
    rp, col, V, Vs, kind = _random_graph(rng)
    T = int(rng.choice([1, 4, 16, 64, 512]))
    c = int(rng.integers(1, 9))
    g = graph(rp, col, num_src=Vs, seg_len=T, block_cost=T + c + int(rng.choice([0, 50, 900])),
              row_cost=c)
    E = len(col)
    print(f"fuzz gated/unfused {case}: {kind} V={V} Vs={Vs} E={E} seg_len={T}", flush=True)
    if Vs == V:  # the gated layer's sources are its destinations
        F, Fe = 64, int(rng.choice([4, 8, 12, 16]))
        H = rng.standard_normal((V, F)).astype(np.float32)
        Ef = rng.standard_normal((E, Fe)).astype(np.float32)
        W_e = (rng.standard_normal((2 * F + Fe, F)) * 0.1).astype(np.float32)
        b_e = rng.standard_normal(F).astype(np.float32)
        Gs = (H.astype(np.float64) @ W_e[:F]).astype(np.float32)
        Gd = (H.astype(np.float64) @ W_e[F:2 * F]).astype(np.float32)
        t = lambda a: dev_padded(a, torch.float32)  # noqa: E731
        Ht, Gst, Gdt = t(H), t(Gs), t(Gd)
        Eft = t(Ef) if E else torch.zeros((0, Fe), device=Ht.device)
        wt = torch.from_numpy(W_e[2 * F:].copy()).to(Ht.device)
        bt = torch.from_numpy(b_e).to(Ht.device)
        extra = dict(gate_src=S.cmat(Gst), gate_dst=S.cmat(Gdt), edge_feat=S.cmat(Eft),
                     w_edge=wt.data_ptr(), gate_bias=bt.data_ptr())
        out = run_gather(g, Ht, dict(msg=S.SAGA_MSG_GATED, reduce=S.SAGA_RED_SUM), F,
                         torch.float32, extra=extra)
        assert rel_err(to_np(out), O.gated_gather(rp, col, H, Ef, W_e, b_e)) <= FP32_TOL
    dtype = str(rng.choice(["f32", "bf16"]))
    Fu = int(rng.choice([1, 8, 41, 128]))
    X = rng.standard_normal((Vs, Fu)).astype(np.float32)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    if dtype == "bf16":
        X = _bf16_round(X)
    for red in ("sum", "max"):
        code = S.SAGA_RED_SUM if red == "sum" else S.SAGA_RED_MAX
        got = to_np(run_unfused(g, dev_padded(X, tdt), dict(reduce=code), Fu, tdt))
        ref = O.gather(rp, col, X, red)
        if red == "max":
            assert np.array_equal(got, ref)
        else:
            assert rel_err(got, ref) <= (FP32_TOL if dtype == "f32" else BF16_TOL)


@pytest.mark.parametrize("case", range(40))
def test_fuzz_layers(case):
    """Whole layers through saga_layer over random graphs and widths: GCN
    (fp32 / bf16, either association order, every activation), SAGE-pool
    and GAT (concatenated or averaged heads)."""
    from paper_2009_00804_amd import layers as LY

    rng = np.random.default_rng(2000 + case)
    rp, col, V = _small_graph(rng, 2500, int(rng.choice([3, 12, 40])),
                              long_row=int(rng.choice([0, 0, 1500])))
    g = graph(rp, col)
    kind = str(rng.choice(["gcn", "sage_pool", "gat"]))
    if kind == "gcn":
        Fi = int(rng.choice([1, 8, 41, 64, 128, 300]))
        Fo = int(rng.choice([1, 16, 41, 64, 128, 200]))
        dtype = str(rng.choice(["f32", "bf16"]))
        act = str(rng.choice(["none", "relu", "elu", "sigmoid", "tanh"]))
        X = rng.standard_normal((V, Fi)).astype(np.float32)
        W = (rng.standard_normal((Fi, Fo)) / np.sqrt(Fi)).astype(np.float32)
        b = rng.standard_normal(Fo).astype(np.float32)
        if dtype == "bf16":
            X, W = _bf16_round(X), _bf16_round(W)
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        print(f"fuzz layer {case}: gcn V={V} E={len(col)} {Fi}->{Fo} {dtype} {act}", flush=True)
        layer = LY.Layer(g, "gcn", Fi, Fo, {"w": W, "b": b}, dtype=tdt, act=act)
        y = to_np(LY.run([layer], dev_padded(X, tdt)))
        tol = FP32_TOL if dtype == "f32" else BF16_TOL
        assert rel_err(y, O.gcn_layer(rp, col, X, W, b, act)) <= tol
    elif kind == "sage_pool":
        F = int(rng.choice([8, 32, 64, 100, 256]))
        Fo = int(rng.choice([8, 64, 256]))
        X = rng.standard_normal((V, F)).astype(np.float32)
        gw = dict(W_pool=(rng.standard_normal((F, F)) / np.sqrt(F)).astype(np.float32),
                  b_pool=rng.standard_normal(F).astype(np.float32),
                  W=(rng.standard_normal((2 * F, Fo)) / np.sqrt(2 * F)).astype(np.float32),
                  b=rng.standard_normal(Fo).astype(np.float32))
        print(f"fuzz layer {case}: sage_pool V={V} E={len(col)} {F}->{Fo}", flush=True)
        y = to_np(LY.run(LY.sage_pool(g, gw), dev_padded(X)))
        want = O.sage_pool_layer(rp, col, X, gw["W_pool"], gw["b_pool"], gw["W"], gw["b"])
        assert rel_err(y, want) <= FP32_TOL
    else:
        H = int(rng.choice([1, 2, 4, 8]))
        D = int(rng.choice([4, 8, 16]))
        Fi = int(rng.choice([16, 64, 512]))
        mean = bool(rng.random() < 0.5)
        X = rng.standard_normal((V, Fi)).astype(np.float32)
        W = (rng.standard_normal((Fi, H * D)) / np.sqrt(Fi)).astype(np.float32)
        al = rng.standard_normal((H, D)).astype(np.float32)
        ar = rng.standard_normal((H, D)).astype(np.float32)
        b = rng.standard_normal(D if mean else H * D).astype(np.float32)
        act = "none" if mean else "elu"
        print(f"fuzz layer {case}: gat V={V} E={len(col)} {Fi}->{H}x{D} mean={mean}", flush=True)
        layer = LY.Layer(g, "gat", Fi, D if mean else H * D,
                         {"w": W, "b": b, "attn_l": al, "attn_r": ar}, heads=H, head_mean=mean,
                         act=act)
        y = to_np(LY.run([layer], dev_padded(X)))
        want = O.gat_layer(rp, col, X, W, al, ar, b, H, "mean" if mean else "concat", act)
        assert rel_err(y, want) <= FP32_TOL


@pytest.mark.parametrize("case", range(40))
def test_fuzz_gather_transform(case):
    """The Gather with the next layer's transform fused in (Sec. 4, cross-stage
    pipelining) over random graphs, plan options, widths of one to four
    whole 128-byte lines, 1 to 64 output columns, split outputs, SUM or MEAN
    with the epilogue, and an optional row scale."""
    import ctypes as C

    from gpu_util import device
    from test_gpu_ops import ACTS, _transform_ref

    S = lib()
    rng = np.random.default_rng(8000 + case)
    rp, col, V, Vs, kind = _random_graph(rng)
    T = int(rng.choice([1, 2, 3, 5, 8, 16, 33, 64, 512]))
    c = int(rng.integers(1, 9))
    B = T + c + int(rng.choice([0, 1, 7, 100, 1000]))
    g = graph(rp, col, num_src=Vs, seg_len=T, block_cost=B, row_cost=c)
    dtype = str(rng.choice(["f32", "bf16"]))
    es = 4 if dtype == "f32" else 2
    F = int(rng.integers(1, 5)) * 128 // es
    N = int(rng.integers(1, 65))
    epv = 16 // es
    split = 0
    if N > epv and rng.random() < 0.5:
        split = int(rng.integers(1, (N - 1) // epv + 1)) * epv
    red = str(rng.choice(["sum", "mean"]))
    dn = int(rng.integers(0, 2))
    act = str(rng.choice(["none", "relu", "tanh"]))
    rsd = rng.integers(0, 50, V).astype(np.int32) if rng.random() < 0.6 else None
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    X = rng.standard_normal((Vs, F)).astype(np.float32)
    W = (rng.standard_normal((F, N)) / np.sqrt(F)).astype(np.float32)
    if dtype == "bf16":
        X, W = _bf16_round(X), _bf16_round(W)
    bias = rng.standard_normal(F)
    print(f"fuzz gather+transform {case}: {kind} V={V} Vs={Vs} seg_len={T} block_cost={B} "
          f"row_cost={c} {dtype} F={F} N={N} split={split} {red} dst_norm={dn} {act} "
          f"row_scale={rsd is not None}", flush=True)
    op = S.saga_edge_op(S.SAGA_MSG_COPY, {"sum": S.SAGA_RED_SUM, "mean": S.SAGA_RED_MEAN}[red],
                        S.dtype_code(tdt), 1, 0, dn, 0.0, ACTS[act])
    Xt, Wt = dev_padded(X, tdt), torch.from_numpy(W).to(tdt).to(device()).contiguous()
    b_t = torch.from_numpy(bias.astype(np.float32)).to(device())
    rs_t = torch.from_numpy(rsd).to(device()) if rsd is not None else None
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(Xt)
    inp.bias = b_t.data_ptr()
    out = dev_padded(np.zeros((V, split if split else N)), dtype=tdt, fill=7.0)
    tail = dev_padded(np.zeros((V, N - split)), dtype=tdt, fill=7.0) if split else None
    nx = S.saga_next_transform()
    nx.w = S.cmat(Wt)
    nx.row_scale_deg = rs_t.data_ptr() if rs_t is not None else None
    nx.split_col = split
    if split:
        nx.tail = S.mat(tail)
    ws = S.workspace(S.saga_gather_transform_workspace_size(g.plan, op, F), device())
    S.saga_scatter_apply_edge_gather_transform(g.plan, op, inp, nx, S.mat(out),
                                               C.c_void_p(ws.data_ptr()), ws.numel(),
                                               S.stream_handle())
    torch.cuda.synchronize()
    got = to_np(out) if not split else np.concatenate([to_np(out), to_np(tail)], axis=1)
    ref, h = _transform_ref(rp, col, X, red, dn, bias, act, Vs, W, rsd, dtype)
    tol = FP32_TOL if dtype == "f32" else BF16_TOL
    assert got.shape == ref.shape
    assert rel_err(got, ref) <= tol
