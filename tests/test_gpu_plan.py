"""Graph layout built on the GPU equals the oracle's, bit for bit."""
import numpy as np
import pytest

from gpu_util import graph, lib
from helpers import FP32_TOL, edges_to_csr, rel_err, tiny_graphs
from oracle import saga_oracle as O

pytestmark = pytest.mark.gpu


def _compare(rp, col, nsrc, T, B, c):
    print(f"plan parity V={len(rp) - 1} E={len(col)} T={T} B={B} c={c}", flush=True)
    g = graph(rp, col, num_src=nsrc, seg_len=T, block_cost=B, row_cost=c)
    got = {k: v.cpu().numpy().astype(np.int64) for k, v in g.arrays().items()}
    want = O.plan(rp, col, nsrc, T, B, c)
    for k in ("d_in", "d_out", "perm", "row_seg_first", "seg_row", "seg_beg", "seg_end",
              "block_ptr"):
        assert np.array_equal(got[k], want[k]), k
    cnt = g.counts
    assert cnt.n_split == want["n_split"]
    assert cnt.s_split == want["row_seg_first"][want["n_split"]]
    assert cnt.num_segments == len(want["seg_row"])
    assert cnt.num_blocks == len(want["block_ptr"]) - 1
    d = np.diff(np.asarray(rp, dtype=np.int64))
    assert cnt.max_in_degree == (d.max() if len(d) else 0)
    assert cnt.error_flags == 0


@pytest.mark.parametrize("case", tiny_graphs(), ids=lambda c: c[0])
@pytest.mark.parametrize("T,B,c", [(2, 6, 1), (3, 16, 4), (512, 4096, 4)])
def test_plan_tiny(case, T, B, c):
    name, n, src, dst = case
    rp, col, _ = edges_to_csr(n, src, dst)
    _compare(rp, col, n, T, B, c)


@pytest.mark.parametrize("T,B,c", [(64, 1024, 4), (512, 4096, 4), (7, 64, 3)])
def test_plan_power_law(T, B, c):
    from synth import configs as C

    g = C.build("sage_rmat", small=True)
    _compare(g["row_ptr"], g["col_idx"], g["num_vertices"], T, B, c)


def test_plan_many_tiles_and_ties():
    """Several radix tiles (V > 2048) with many equal degrees."""
    rng = np.random.default_rng(3)
    V = 20000
    deg = rng.integers(0, 5, V)
    deg[rng.integers(0, V, 30)] = rng.integers(600, 3000, 30)
    rp = np.concatenate([[0], np.cumsum(deg)]).astype(np.int64)
    col = rng.integers(0, V, rp[-1])
    _compare(rp, col, V, 512, 4096, 4)
    _compare(rp, col, V, 16, 256, 1)


@pytest.mark.parametrize("nsrc", [(1 << 23) - 5, 1 << 23, (1 << 23) + 1],
                         ids=["below", "at", "past"])
def test_plan_source_count_limit(nsrc):
    """The bucketed out-degree count takes up to 2^23 sources; past that the
    degree kernel counts with atomics.  Both sides of the boundary, with the
    first and last source ids, a hub source and a ragged last edge tile."""
    rng = np.random.default_rng(11)
    V = 3000
    deg = rng.integers(0, 60, V)
    deg[:3] = 7000
    rp = np.concatenate([[0], np.cumsum(deg)]).astype(np.int64)
    E = int(rp[-1])
    col = rng.integers(0, nsrc, E)
    col[:40] = nsrc - 1
    col[40:80] = 0
    col[rng.choice(E, 20000, replace=False)] = nsrc // 3
    assert E % 16384 != 0
    _compare(rp, col, nsrc, 512, 4096, 4)


def test_plan_edge_cases():
    # no edges at all
    _compare(np.zeros(6, np.int64), np.zeros(0, np.int64), 5, 4, 8, 1)
    # one vertex, one self-loop
    _compare(np.array([0, 1]), np.array([0]), 1, 4, 8, 1)
    # a single row longer than many segments; more sources than destinations
    _compare(np.array([0, 0, 1000, 1000]), np.arange(1000) % 7, 7, 16, 64, 2)


def test_plan_rejects_invalid_csr():
    """Errors found by the device validation are reported, and the later
    kernels skip their work instead of reading out of bounds."""
    S = lib()
    cases = [
        (np.array([1, 2, 3]), np.array([0, 1, 0]), 1),       # row_ptr[0] != 0
        (np.array([0, 3, 2, 4]), np.array([0, 1, 2, 0]), 2),  # decreasing
        (np.array([0, 1, 2]), np.array([0, 1, 1]), 4),       # row_ptr[V] != E
        (np.array([0, 1, 3]), np.array([0, 5, 1]), 8),       # col out of range
    ]
    for rp, col, bit in cases:
        g = graph(rp, col, check=False)
        st, counts = S.saga_plan_check(g.plan, S.stream_handle())
        assert st == S.SAGA_EGRAPH
        assert counts.error_flags & bit


def test_split_plan_equals_single_stream_plan_and_overlaps_the_transform():
    """saga_plan_build_split (out-degree branch on the stream, row order on a
    second stream) gives the oracle's plan bit for bit (and so the arrays of
    saga_plan_build), and the GCN layer whose transform is enqueued between
    the branches matches the oracle's layer (and the sequential order's
    bytes)."""
    import ctypes as C

    import torch

    from gpu_util import dev_int, device, lib, to_np
    from synth import configs as Cfg
    from paper_2009_00804_amd import layers as LY

    S = lib()
    g = Cfg.build("gcn_rmat", small=True)
    V, E = g["num_vertices"], g["num_edges"]
    print(f"split plan V={V} E={E}", flush=True)
    rp, col = dev_int(g["row_ptr"]), dev_int(g["col_idx"])
    ref = S.Graph(rp, col)
    want = {k: v.cpu().numpy() for k, v in ref.arrays().items()}
    p0 = ref.plan
    oracle = O.plan(g["row_ptr"], g["col_idx"], V, p0.seg_len, p0.block_cost, p0.row_cost)
    main = torch.cuda.current_stream()
    side = torch.cuda.Stream()
    fork, join = torch.cuda.Event(), torch.cuda.Event()
    fork.record(main)
    join.record(main)  # creates both events
    for _ in range(2):  # twice, each into a workspace filled with garbage
        ws = torch.full((ref.ws.numel(),), 0xAB, dtype=torch.uint8, device=device())
        plan = S.saga_plan_build_split(V, V, E, C.c_void_p(rp.data_ptr()), C.c_void_p(col.data_ptr()),
                                       ref.opts, C.c_void_p(ws.data_ptr()), ws.numel(),
                                       S.stream_handle(main), S.stream_handle(side),
                                       C.c_void_p(fork.cuda_event), C.c_void_p(join.cuda_event))
        main.wait_event(join)
        st, counts = S.saga_plan_check(plan, S.stream_handle(main))
        assert st == S.SAGA_OK
        gr = S.Graph.__new__(S.Graph)
        gr.__dict__.update(ref.__dict__)
        gr.plan, gr.ws, gr.counts = plan, ws, counts
        got = {k: v.cpu().numpy() for k, v in gr.arrays().items()}
        for k in want:
            assert np.array_equal(got[k].astype(np.int64), oracle[k].astype(np.int64)), k
            assert np.array_equal(got[k], want[k]), k
        assert counts.n_split == oracle["n_split"]
    # layer 1 of the GCN with its transform enqueued between the branches
    X = torch.from_numpy(np.ascontiguousarray(g["X"][:, :g["dims"][0]])).to(device())
    X = torch.nn.functional.pad(X, (0, (-X.shape[1]) % 4))[:, :g["dims"][0]]
    W1 = torch.from_numpy(g["W1"]).to(device())
    b1 = torch.from_numpy(g["b1"]).to(device())
    F = W1.shape[1]
    none = S.saga_cmat(None, 0, 0, 0)

    def layer1(pl, wait=None):
        Z = torch.empty((V, F), device=device())
        H = torch.empty((V, F), device=device())
        gop = S.saga_gemm_op(S.SAGA_F32, S.SAGA_GEMM_PLAIN, S.SAGA_ACT_NONE, pl.d_out)
        mws = S.workspace(S.saga_apply_vertex_workspace_size(gop, X.shape[1], 0, F), device())
        S.saga_apply_vertex(gop, S.cmat(X), S.cmat(W1), none, none, None, None, S.mat(Z),
                            C.c_void_p(mws.data_ptr()), mws.numel(), S.stream_handle(main))
        if wait is not None:
            main.wait_event(wait)
        op = S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 1, 0.0, S.SAGA_ACT_RELU)
        inp = S.saga_edge_inputs()
        inp.src = S.cmat(Z)
        inp.bias = b1.data_ptr()
        gws = S.workspace(S.saga_gather_workspace_size(pl, op, F), device())
        S.saga_scatter_apply_edge_gather(pl, op, inp, S.mat(H), C.c_void_p(gws.data_ptr()), gws.numel(),
                                         S.stream_handle(main))
        torch.cuda.synchronize()
        return to_np(H)

    seq = layer1(ref.plan)
    ws2 = torch.empty_like(ref.ws)
    plan2 = S.saga_plan_build_split(V, V, E, C.c_void_p(rp.data_ptr()), C.c_void_p(col.data_ptr()),
                                    ref.opts, C.c_void_p(ws2.data_ptr()), ws2.numel(),
                                    S.stream_handle(main), S.stream_handle(side),
                                    C.c_void_p(fork.cuda_event), C.c_void_p(join.cuda_event))
    piped = layer1(plan2, wait=join)
    ref1 = O.gcn_layer(g["row_ptr"], g["col_idx"], g["X"][:, :g["dims"][0]], g["W1"], g["b1"], "relu")
    assert rel_err(piped, ref1) <= FP32_TOL
    assert np.array_equal(piped, seq)
    with pytest.raises(S.SagaError):
        S.saga_plan_build_split(V, V, E, C.c_void_p(rp.data_ptr()), C.c_void_p(col.data_ptr()),
                                ref.opts, C.c_void_p(ws.data_ptr()), ws.numel(),
                                S.stream_handle(main), S.stream_handle(main),
                                C.c_void_p(fork.cuda_event), C.c_void_p(join.cuda_event))
