"""The C-ABI library on the host (no GPU needed): it loads, exports every
entry point include/saga.h declares, and rejects bad arguments before any
kernel is launched."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def S():
    import paper_2009_00804_amd.saga as S

    if not os.path.exists(S.LIB_PATH):
        from paper_2009_00804_amd import build

        build.build()
    S.lib()
    return S


def test_missing_library_raises_no_fallback(tmp_path):
    """Without libsaga.so the binding raises at the first call: no op has a
    CPU or PyTorch fallback."""
    import paper_2009_00804_amd.saga as S

    saved_path, saved_lib = S.LIB_PATH, S._lib
    try:
        S.LIB_PATH = str(tmp_path / "libsaga.so")
        S._lib = None
        with pytest.raises(RuntimeError, match="not built"):
            S.lib()
    finally:
        S.LIB_PATH, S._lib = saved_path, saved_lib


def _declared():
    src = open(os.path.join(ROOT, "include", "saga.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(saga_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = _declared()
    for want in ("saga_plan_build", "saga_scatter_apply_edge_gather", "saga_apply_vertex",
                 "saga_layer"):
        assert want in names


def test_library_exports_every_declared_symbol(S):
    L = S.lib()
    for name in _declared():
        assert hasattr(L, name), name
    assert sorted(S.EXPORTS) == _declared()


def test_version_and_status_strings(S):
    assert "gfx950" in S.saga_version()
    L = S.lib()
    assert L.saga_status_str(S.SAGA_OK) == b"ok"
    assert L.saga_status_str(S.SAGA_EGRAPH) == b"invalid graph"


def test_error_detail_is_per_thread(S):
    """saga_last_error is thread-local: two threads that fail in different
    ways each read back their own detail, and a success in one thread
    clears only that thread's."""
    import threading

    L = S.lib()
    bar = threading.Barrier(2)
    seen = {}

    def worker(name, fail):
        fail()
        bar.wait()  # both threads have failed before either reads
        seen[name] = L.saga_last_error().decode()
        bar.wait()
        if name == "a":
            assert L.saga_plan_workspace_size(10, 10, 5, None, C.byref(C.c_size_t())) == S.SAGA_OK
        bar.wait()
        seen[name + "2"] = L.saga_last_error().decode()

    out = C.c_size_t()
    ta = threading.Thread(target=worker, args=("a", lambda: L.saga_plan_workspace_size(
        10, 10, -1, None, C.byref(out))))
    tb = threading.Thread(target=worker, args=("b", lambda: L.saga_plan_workspace_size(
        10, 10, 5, None, None)))
    ta.start(); tb.start(); ta.join(); tb.join()
    assert "out of range" in seen["a"] and "null" in seen["b"], seen
    assert seen["a2"] == "" and seen["b2"] == seen["b"], seen


def test_plan_workspace_size_rules(S):
    n = S.saga_plan_workspace_size(1000, 1000, 5000)
    assert n > 0 and n % 256 == 0
    assert S.saga_plan_workspace_size(0, 0, 0) >= 0
    for args, opts in [((10, 10, -1), None), ((10, 10, 1 << 31), None),
                       ((10, 10, 5), S.saga_plan_opts(64, 32, 4))]:
        with pytest.raises(S.SagaError) as e:
            S.saga_plan_workspace_size(*args, opts)
        assert e.value.status == S.SAGA_EINVAL


def test_plan_edge_limit(S):
    """The largest graph a plan takes: every int32 edge offset and segment
    cost prefix must fit, so the limit depends on num_dst, seg_len and
    row_cost; one edge more is refused before anything is allocated."""
    from helpers import plan_edge_limit

    for V, T, c in [(1 << 21, 512, 4), (1000, 64, 1), (1 << 27, 4096, 8), (0, 512, 4)]:
        opts = S.saga_plan_opts(T, T + c, c)
        E = plan_edge_limit(V, T, c)
        assert S.saga_plan_workspace_size(V, V, E, opts) > 0
        with pytest.raises(S.SagaError) as e:
            S.saga_plan_workspace_size(V, V, E + 1, opts)
        assert e.value.status == S.SAGA_EINVAL


def test_plan_build_rejects_bad_arguments_without_launching(S):
    ws = C.create_string_buffer(1 << 16)
    with pytest.raises(S.SagaError) as e:
        S.saga_plan_build(10, 10, 5, None, None, None, C.addressof(ws), 1 << 16, None)
    assert e.value.status == S.SAGA_EINVAL
    with pytest.raises(S.SagaError) as e:   # workspace too small
        S.saga_plan_build(10, 10, 5, 1024, 2048, None, 4096, 16, None)
    assert e.value.status == S.SAGA_EWORKSPACE


def _fake_plan(S, V=16, E=40):
    p = S.saga_plan()
    p.num_dst = p.num_src = V
    p.num_edges = E
    p.row_ptr, p.col_idx = 0x10000, 0x20000
    for f in ("d_in", "d_out", "perm", "row_seg_first", "seg_row", "seg_beg", "seg_end",
              "block_ptr", "counts"):
        setattr(p, f, 0x30000)
    p.max_split_segments = 0
    return p


def test_gather_rejects_bad_arguments(S):
    p = _fake_plan(S)
    op = S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 0, 0.2, 0)
    inp = S.saga_edge_inputs()
    out = S.saga_mat(0x40000, 16, 8, 8)
    L = S.lib()

    def call(o=op, i=inp, ou=out):
        return L.saga_scatter_apply_edge_gather(C.byref(p), C.byref(o), C.byref(i), ou, None, 0, None)

    inp.src = S.saga_cmat(0x50000, 16, 8, 8)
    # wrong source shape
    inp.src = S.saga_cmat(0x50000, 15, 8, 8)
    assert call() == S.SAGA_EINVAL
    # ld < cols
    inp.src = S.saga_cmat(0x50000, 16, 8, 4)
    assert call() == S.SAGA_EINVAL
    # misaligned base
    inp.src = S.saga_cmat(0x50004, 16, 8, 8)
    assert call() == S.SAGA_EINVAL
    # row pitch not a multiple of 16 bytes
    inp.src = S.saga_cmat(0x50000, 16, 3, 3)
    assert call(ou=S.saga_mat(0x40000, 16, 3, 4)) == S.SAGA_EINVAL
    inp.src = S.saga_cmat(0x50000, 16, 8, 8)
    # output overlapping the source
    assert call(ou=S.saga_mat(0x50000 + 64, 16, 8, 8)) == S.SAGA_EINVAL
    # unsupported combinations
    bad = S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_SOFTMAX, S.SAGA_F32, 1, 0, 0, 0.2, 0)
    assert call(o=bad) == S.SAGA_EUNSUPPORTED
    bad = S.saga_edge_op(S.SAGA_MSG_GAT, S.SAGA_RED_SOFTMAX, S.SAGA_BF16, 2, 0, 0, 0.2, 0)
    inp.src = S.saga_cmat(0x50000, 16, 8, 8)
    assert call(o=bad) == S.SAGA_EUNSUPPORTED
    bad = S.saga_edge_op(S.SAGA_MSG_GAT, S.SAGA_RED_SOFTMAX, S.SAGA_F32, 3, 0, 0, 0.2, 0)
    assert call(o=bad) == S.SAGA_EUNSUPPORTED   # 3 heads do not divide 8 columns
    bad = S.saga_edge_op(S.SAGA_MSG_GATED, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 0, 0.2, 0)
    assert call(o=bad) == S.SAGA_EUNSUPPORTED   # gated needs F == 64
    assert b"F == 64" in L.saga_last_error()


def test_trace_stages_rejects_bad_arguments(S):
    L = S.lib()
    assert L.saga_trace_stages(None, -1, 0) == S.SAGA_EINVAL
    assert L.saga_trace_stages(None, 2, 0) == S.SAGA_EINVAL
    arr = (C.c_void_p * 2)(None, None)
    assert L.saga_trace_stages(arr, 2, 1) == S.SAGA_EINVAL     # null events
    assert L.saga_trace_stages(None, 0, 0) == S.SAGA_OK         # tracing off


def test_gather_transform_rejects_unsupported_shapes(S):
    p = _fake_plan(S)
    L = S.lib()
    inp = S.saga_edge_inputs()
    inp.src = S.saga_cmat(0x50000, 16, 32, 32)          # one 128-byte line of float32
    nx = S.saga_next_transform()
    nx.w = S.saga_cmat(0x70000, 32, 8, 8)
    out = S.saga_mat(0x40000, 16, 8, 8)
    ws, wsb = C.c_void_p(0x100000), 1 << 20

    def call(op, ou=out):
        return L.saga_scatter_apply_edge_gather_transform(C.byref(p), C.byref(op), C.byref(inp),
                                                          C.byref(nx), ou, ws, wsb, None)

    sum_op = S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 0, 0.2, 0)
    assert call(S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_MAX, S.SAGA_F32, 1, 0, 0, 0.2, 0)) \
        == S.SAGA_EUNSUPPORTED
    inp.src = S.saga_cmat(0x50000, 16, 24, 24)           # not whole 128-byte lines
    assert call(sum_op) == S.SAGA_EUNSUPPORTED
    inp.src = S.saga_cmat(0x50000, 16, 32, 32)
    nx.w = S.saga_cmat(0x70000, 32, 65, 65)               # more than 64 outputs
    assert call(sum_op, ou=S.saga_mat(0x40000, 16, 65, 68)) == S.SAGA_EUNSUPPORTED
    nx.w = S.saga_cmat(0x70000, 32, 8, 12)                # weights not dense
    assert call(sum_op) == S.SAGA_EINVAL
    nx.w = S.saga_cmat(0x70000, 32, 8, 8)
    nx.split_col = 2                                      # split inside a 16-byte vector
    assert call(sum_op, ou=S.saga_mat(0x40000, 16, 2, 4)) == S.SAGA_EINVAL
    nx.split_col = 0
    assert call(sum_op, ou=S.saga_mat(0x70000 + 16, 16, 8, 8)) == S.SAGA_EINVAL   # out on w


def test_unfused_rejects_bad_arguments(S):
    """The unfused baseline: unsupported ops, workspace size, alignment and
    overlap are all rejected on the host before any launch."""
    p = _fake_plan(S)
    op = S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 0, 0.2, 0)
    inp = S.saga_edge_inputs()
    inp.src = S.saga_cmat(0x50000, 16, 8, 8)
    out = S.saga_mat(0x40000, 16, 8, 8)
    L = S.lib()

    def call(o=op, ws=0x900000, nb=1 << 20):
        return L.saga_scatter_gather_unfused(C.byref(p), C.byref(o), C.byref(inp), out, ws, nb, None)

    need = S.saga_unfused_workspace_size(p, op, 8)
    assert need >= 40 * 8 * 4      # the E x F edge tensor
    big = S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 0, 0.2, 0)
    assert S.saga_unfused_workspace_size(p, big, 64) > need
    assert call(nb=need - 1) == S.SAGA_EWORKSPACE
    assert call(ws=None, nb=0) == S.SAGA_EWORKSPACE
    assert call(ws=0x900000 + 16, nb=need) == S.SAGA_EINVAL        # not 256-byte aligned
    assert call(ws=0x40000, nb=need) == S.SAGA_EINVAL              # overlaps the output
    gat = S.saga_edge_op(S.SAGA_MSG_GAT, S.SAGA_RED_SOFTMAX, S.SAGA_F32, 2, 0, 0, 0.2, 0)
    assert call(o=gat) == S.SAGA_EUNSUPPORTED
    soft = S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_SOFTMAX, S.SAGA_F32, 1, 0, 0, 0.2, 0)
    assert call(o=soft) == S.SAGA_EUNSUPPORTED
    gated = S.saga_edge_op(S.SAGA_MSG_GATED, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 0, 0.2, 0)
    assert call(o=gated) == S.SAGA_EUNSUPPORTED


def test_lstm_gather_rejects_bad_arguments(S):
    p = _fake_plan(S)
    L = S.lib()
    gx = S.saga_cmat(0x50000, 16, 512, 512)
    whh = S.saga_cmat(0x90000, 128, 512, 512)
    out = S.saga_mat(0x100000, 16, 128, 128)

    def call(g=gx, w=whh, o=out, ws=0x900000, nb=256):
        return L.saga_lstm_gather(C.byref(p), g, w, o, ws, nb, None)

    assert S.saga_lstm_gather_workspace_size(p, 128) == 256
    assert L.saga_lstm_gather_workspace_size(C.byref(p), 100, C.byref(C.c_size_t())) == S.SAGA_EUNSUPPORTED
    assert call(w=S.saga_cmat(0x90000, 100, 400, 400)) == S.SAGA_EUNSUPPORTED    # H = 100
    assert call(g=S.saga_cmat(0x50000, 15, 512, 512)) == S.SAGA_EINVAL           # rows != num_src
    assert call(g=S.saga_cmat(0x50000, 16, 256, 256)) == S.SAGA_EINVAL           # not 4H columns
    assert call(o=S.saga_mat(0x100000, 16, 64, 64)) == S.SAGA_EINVAL             # not H columns
    assert call(nb=8) == S.SAGA_EWORKSPACE
    assert call(ws=0x900010) == S.SAGA_EINVAL                                   # misaligned
    assert call(o=S.saga_mat(0x50000 + 256, 16, 128, 128)) == S.SAGA_EINVAL      # overlaps gates_x
    rows = lambda b, e: L.saga_lstm_gather_rows(C.byref(p), b, e, gx, whh, out, 0x900000, 256,  # noqa: E731
                                                 None)
    assert rows(-1, 4) == S.SAGA_EINVAL
    assert rows(5, 4) == S.SAGA_EINVAL
    assert rows(0, 17) == S.SAGA_EINVAL                                          # past num_dst


def test_gemm_rejects_bad_arguments(S):
    L = S.lib()
    op = S.saga_gemm_op(S.SAGA_F32, S.SAGA_GEMM_PLAIN, 0, None)
    a = S.saga_cmat(0x10000, 100, 32, 32)
    w = S.saga_cmat(0x20000, 32, 16, 16)
    none = S.saga_cmat(None, 0, 0, 0)
    out = S.saga_mat(0x30000, 100, 16, 16)
    f = lambda *args: L.saga_apply_vertex(C.byref(args[0]), *args[1:])  # noqa: E731
    assert f(op, a, S.saga_cmat(0x20000, 31, 16, 16), none, none, None, None, out, 0x900000, 1 << 20, None) == S.SAGA_EINVAL
    assert f(op, a, w, none, none, None, None, S.saga_mat(0x30000, 99, 16, 16), 0x900000, 1 << 20, None) == S.SAGA_EINVAL
    assert f(op, a, w, none, none, None, None, S.saga_mat(0x10000 + 128, 100, 16, 16), 0x900000, 1 << 20, None) == S.SAGA_EINVAL
    gru = S.saga_gemm_op(S.SAGA_F32, S.SAGA_GEMM_GRU, 0, None)
    w3 = S.saga_cmat(0x20000, 32, 60, 60)
    a2 = S.saga_cmat(0x60000, 100, 20, 20)
    w23 = S.saga_cmat(0x70000, 20, 60, 60)
    assert f(gru, a, w3, a2, w23, None, None, S.saga_mat(0x30000, 100, 20, 20), 0x900000, 1 << 20, None) == S.SAGA_EUNSUPPORTED
    bad_mode = S.saga_gemm_op(S.SAGA_F32, 7, 0, None)
    assert f(bad_mode, a, w, none, none, None, None, out, 0x900000, 1 << 20, None) == S.SAGA_EINVAL


def test_layer_rejects_bad_descriptors(S):
    p = _fake_plan(S)
    L = S.lib()
    d = S.saga_layer_desc()
    d.kind = S.SAGA_LAYER_GAT
    d.dtype = S.SAGA_BF16
    d.in_feat, d.out_feat, d.heads = 8, 8, 2
    d.w = d.attn_l = d.attn_r = 0x1000
    n = C.c_size_t()
    assert L.saga_layer_workspace_size(C.byref(p), C.byref(d), C.byref(n)) == S.SAGA_EUNSUPPORTED
    # the other float32-only kinds refuse bf16 the same way
    for kind in (S.SAGA_LAYER_SAGE_POOL, S.SAGA_LAYER_SAGE_LSTM, S.SAGA_LAYER_GATED_GRU):
        e = S.saga_layer_desc()
        e.kind, e.dtype, e.in_feat, e.out_feat, e.hidden = kind, S.SAGA_BF16, 8, 8, 32
        e.w = e.w_pool = e.w_ih = e.w_hh = e.w_e = 0x1000
        assert L.saga_layer_workspace_size(C.byref(p), C.byref(e), C.byref(n)) == S.SAGA_EUNSUPPORTED
    d.kind = 9
    assert L.saga_layer_workspace_size(C.byref(p), C.byref(d), C.byref(n)) == S.SAGA_EINVAL
    d.kind = S.SAGA_LAYER_GCN
    d.dtype = S.SAGA_F32
    assert L.saga_layer_workspace_size(C.byref(p), C.byref(d), C.byref(n)) == S.SAGA_OK
    assert n.value > 0
    # workspace missing
    x = S.saga_cmat(0x50000, 16, 8, 8)
    out = S.saga_mat(0x60000, 16, 8, 8)
    none = S.saga_cmat(None, 0, 0, 0)
    assert L.saga_layer(C.byref(p), C.byref(d), x, none, out, None, 0, None) == S.SAGA_EWORKSPACE


def _fake_rel(S, p, R=4):
    r = S.saga_rel_plan()
    r.num_rel, r.num_src, r.num_edges = R, p.num_src, p.num_edges
    r.max_pairs = 256
    r.etype = 0x70000
    r.plan_counts = p.counts
    for f in ("rel_ptr", "rel_count", "pair_src", "edge_pair", "edge_norm", "counts"):
        setattr(r, f, 0x80000)
    return r


def test_rel_plan_rejects_bad_arguments(S):
    p = _fake_plan(S)
    L = S.lib()
    n = S.saga_rel_plan_workspace_size(p, 4)
    assert n > 0 and n % 256 == 0
    assert S.saga_rel_plan_workspace_size(p, S.SAGA_REL_MAX_RELATIONS) > n
    sz = C.c_size_t()
    for R in (0, -1, S.SAGA_REL_MAX_RELATIONS + 1):
        assert L.saga_rel_plan_workspace_size(C.byref(p), R, C.byref(sz)) == S.SAGA_EINVAL
    rel = S.saga_rel_plan()

    def build(et=0x70000, R=4, ws=0x1000000, nb=n):
        return L.saga_rel_plan_build(C.byref(p), et, R, ws, nb, None, C.byref(rel))

    assert build(et=None) == S.SAGA_EINVAL
    assert build(R=0) == S.SAGA_EINVAL
    assert build(nb=n - 1) == S.SAGA_EWORKSPACE
    assert build(ws=0x1000010) == S.SAGA_EINVAL                    # misaligned
    assert build(ws=0x70000 - 256, nb=n) == S.SAGA_EINVAL          # overlaps etype
    unbuilt = S.saga_plan()
    assert L.saga_rel_plan_build(C.byref(unbuilt), 0x70000, 4, 0x1000000, n, None,
                                 C.byref(rel)) == S.SAGA_EINVAL


def test_rel_transform_rejects_bad_arguments(S):
    p = _fake_plan(S)
    r = _fake_rel(S, p)
    L = S.lib()
    need = S.saga_rel_transform_workspace_size(r, S.SAGA_F32, 32, 16)
    assert need > 0
    x = S.saga_cmat(0x100000, 16, 32, 32)
    w = S.saga_cmat(0x200000, 4 * 32, 16, 16)
    out = S.saga_mat(0x300000, 256, 16, 16)

    def call(x=x, w=w, o=out, ws=0x900000, nb=need, dt=S.SAGA_F32):
        return L.saga_rel_transform(C.byref(r), dt, x, w, o, ws, nb, None)

    assert call(w=S.saga_cmat(0x200000, 3 * 32, 16, 16)) == S.SAGA_EINVAL   # not num_rel stacked
    assert call(x=S.saga_cmat(0x100000, 15, 32, 32)) == S.SAGA_EINVAL       # rows != num_src
    assert call(o=S.saga_mat(0x300000, 255, 16, 16)) == S.SAGA_EINVAL       # rows != max_pairs
    assert call(nb=need - 1) == S.SAGA_EWORKSPACE
    assert call(ws=0x900010) == S.SAGA_EINVAL
    assert call(o=S.saga_mat(0x100000 + 256, 256, 16, 16)) == S.SAGA_EINVAL  # overlaps x
    assert call(dt=5) == S.SAGA_EINVAL
    assert L.saga_rel_transform(None, S.SAGA_F32, x, w, out, 0x900000, need, None) == S.SAGA_EINVAL


def test_typed_gather_and_layer_reject_bad_arguments(S):
    p = _fake_plan(S)
    r = _fake_rel(S, p)
    L = S.lib()
    op = S.saga_edge_op(S.SAGA_MSG_TYPED, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 0, 0.0, 0)
    inp = S.saga_edge_inputs()
    inp.src = S.saga_cmat(0x100000, 256, 8, 8)
    out = S.saga_mat(0x400000, 16, 8, 8)

    def call(o=op):
        return L.saga_scatter_apply_edge_gather(C.byref(p), C.byref(o), C.byref(inp), out, None, 0,
                                                None)

    assert call() == S.SAGA_EINVAL                       # no rel plan
    inp.rel = C.pointer(r)
    mean = S.saga_edge_op(S.SAGA_MSG_TYPED, S.SAGA_RED_MEAN, S.SAGA_F32, 1, 0, 0, 0.0, 0)
    assert call(o=mean) == S.SAGA_EUNSUPPORTED
    inp.src = S.saga_cmat(0x100000, 16, 8, 8)            # rows must be max_pairs
    assert call() == S.SAGA_EINVAL
    inp.src = S.saga_cmat(0x100000, 256, 8, 8)
    other = _fake_rel(S, p)
    other.plan_counts = 0x31000                          # built on another plan
    inp.rel = C.pointer(other)
    assert call() == S.SAGA_EINVAL
    inp.rel = C.pointer(r)
    inp.self = S.saga_cmat(0x500000, 15, 8, 8)           # self rows != num_dst
    assert call() == S.SAGA_EINVAL
    inp.self = S.saga_cmat(0x400000 + 64, 16, 8, 8)      # overlaps out
    assert call() == S.SAGA_EINVAL
    # the layer needs w, w_self and a rel plan of the same graph
    d = S.saga_layer_desc()
    d.kind = S.SAGA_LAYER_RGCN
    d.dtype = S.SAGA_F32
    d.in_feat, d.out_feat = 8, 8
    d.w = 0x1000
    n = C.c_size_t()
    assert L.saga_layer_workspace_size(C.byref(p), C.byref(d), C.byref(n)) == S.SAGA_EINVAL
    d.w_self = 0x2000
    assert L.saga_layer_workspace_size(C.byref(p), C.byref(d), C.byref(n)) == S.SAGA_EINVAL
    d.rel = C.pointer(r)
    assert L.saga_layer_workspace_size(C.byref(p), C.byref(d), C.byref(n)) == S.SAGA_OK
    assert n.value > 0
