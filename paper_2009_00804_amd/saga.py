"""ctypes binding of libsaga.so (include/saga.h).

The ``saga_*`` functions here have the names and arguments of the C entry
points and only marshal arguments; every stage of the layer runs in the HIP
kernels of the library.  torch supplies device memory and the stream.  If the
library is missing this module raises at import of the library (there is no
fallback path).

Convenience wrappers (``Graph``, ``cmat``, ``mat``) build the C structs from
torch tensors and allocate workspaces with torch.
"""
from __future__ import annotations

import ctypes as C
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libsaga.so")

# enums (saga.h)
SAGA_OK, SAGA_EINVAL, SAGA_EGRAPH, SAGA_EUNSUPPORTED, SAGA_EDEVICE, SAGA_EWORKSPACE, SAGA_EINTERNAL = range(7)
SAGA_F32, SAGA_BF16 = 0, 1
SAGA_RED_SUM, SAGA_RED_MEAN, SAGA_RED_MAX, SAGA_RED_SOFTMAX = range(4)
SAGA_MSG_COPY, SAGA_MSG_SRC_NORM, SAGA_MSG_GAT, SAGA_MSG_GATED, SAGA_MSG_TYPED = range(5)
SAGA_ACT_NONE, SAGA_ACT_RELU, SAGA_ACT_ELU, SAGA_ACT_SIGMOID, SAGA_ACT_TANH = range(5)
SAGA_GEMM_PLAIN, SAGA_GEMM_CONCAT, SAGA_GEMM_GRU = range(3)
(SAGA_LAYER_GCN, SAGA_LAYER_GAT, SAGA_LAYER_SAGE_POOL, SAGA_LAYER_GATED_GRU, SAGA_LAYER_SAGE_LSTM,
 SAGA_LAYER_RGCN) = range(6)
SAGA_REL_TILE = 128
SAGA_REL_MAX_RELATIONS = 2048

ACT = {"none": 0, "relu": 1, "elu": 2, "sigmoid": 3, "tanh": 4}

EXPORTS = [
    "saga_plan_workspace_size", "saga_plan_build", "saga_plan_build_split", "saga_plan_check",
    "saga_gather_workspace_size", "saga_scatter_apply_edge_gather",
    "saga_scatter_apply_edge_gather_noalloc", "saga_gather_transform_workspace_size",
    "saga_scatter_apply_edge_gather_transform",
    "saga_unfused_workspace_size", "saga_scatter_gather_unfused",
    "saga_lstm_gather_workspace_size", "saga_lstm_gather", "saga_lstm_gather_rows",
    "saga_rel_plan_workspace_size", "saga_rel_plan_build", "saga_rel_plan_check",
    "saga_rel_transform_workspace_size", "saga_rel_transform",
    "saga_apply_vertex_workspace_size", "saga_apply_vertex",
    "saga_layer_workspace_size", "saga_layer", "saga_trace_stages", "saga_sync_check",
    "saga_status_str", "saga_last_error", "saga_version",
]


class saga_cmat(C.Structure):
    _fields_ = [("ptr", C.c_void_p), ("rows", C.c_int64), ("cols", C.c_int64), ("ld", C.c_int64)]


class saga_mat(C.Structure):
    _fields_ = [("ptr", C.c_void_p), ("rows", C.c_int64), ("cols", C.c_int64), ("ld", C.c_int64)]


class saga_plan_opts(C.Structure):
    _fields_ = [("seg_len", C.c_int32), ("block_cost", C.c_int32), ("row_cost", C.c_int32)]


class saga_plan(C.Structure):
    _fields_ = [
        ("num_dst", C.c_int32), ("num_src", C.c_int32), ("num_edges", C.c_int64),
        ("row_ptr", C.c_void_p), ("col_idx", C.c_void_p),
        ("seg_len", C.c_int32), ("block_cost", C.c_int32), ("row_cost", C.c_int32),
        ("max_segments", C.c_int64), ("max_blocks", C.c_int64), ("max_split", C.c_int64),
        ("max_split_segments", C.c_int64),
        ("d_in", C.c_void_p), ("d_out", C.c_void_p), ("perm", C.c_void_p),
        ("row_seg_first", C.c_void_p), ("seg_row", C.c_void_p), ("seg_beg", C.c_void_p),
        ("seg_end", C.c_void_p), ("block_ptr", C.c_void_p), ("counts", C.c_void_p),
        ("scratch", C.c_void_p), ("scratch_bytes", C.c_size_t),
    ]


class saga_plan_counts(C.Structure):
    _fields_ = [("num_segments", C.c_int64), ("num_blocks", C.c_int64), ("n_split", C.c_int64),
                ("s_split", C.c_int64), ("error_flags", C.c_int32), ("max_in_degree", C.c_int32)]


class saga_rel_plan(C.Structure):
    _fields_ = [
        ("num_rel", C.c_int32), ("num_src", C.c_int32), ("num_edges", C.c_int64),
        ("max_pairs", C.c_int64), ("etype", C.c_void_p), ("plan_counts", C.c_void_p),
        ("rel_ptr", C.c_void_p), ("rel_count", C.c_void_p), ("pair_src", C.c_void_p),
        ("edge_pair", C.c_void_p), ("edge_norm", C.c_void_p), ("counts", C.c_void_p),
        ("scratch", C.c_void_p), ("scratch_bytes", C.c_size_t),
    ]


class saga_rel_counts(C.Structure):
    _fields_ = [("pair_rows", C.c_int64), ("pairs", C.c_int64), ("error_flags", C.c_int32)]


class saga_edge_op(C.Structure):
    _fields_ = [("msg", C.c_int), ("reduce", C.c_int), ("dtype", C.c_int), ("heads", C.c_int32),
                ("head_mean", C.c_int32), ("dst_norm", C.c_int32), ("neg_slope", C.c_float),
                ("act", C.c_int)]


class saga_edge_inputs(C.Structure):
    _fields_ = [("src", saga_cmat), ("el", saga_cmat), ("er", saga_cmat), ("gate_src", saga_cmat),
                ("gate_dst", saga_cmat), ("edge_feat", saga_cmat), ("w_edge", C.c_void_p),
                ("gate_bias", C.c_void_p), ("bias", C.c_void_p), ("rel", C.POINTER(saga_rel_plan)),
                ("self", saga_cmat)]


class saga_next_transform(C.Structure):
    _fields_ = [("w", saga_cmat), ("row_scale_deg", C.c_void_p), ("split_col", C.c_int32),
                ("tail", saga_mat)]


class saga_gemm_op(C.Structure):
    _fields_ = [("dtype", C.c_int), ("mode", C.c_int), ("act", C.c_int),
                ("row_scale_deg", C.c_void_p), ("split_col", C.c_int32), ("tail", saga_mat)]


class saga_layer_desc(C.Structure):
    _fields_ = [
        ("kind", C.c_int), ("dtype", C.c_int), ("in_feat", C.c_int32), ("out_feat", C.c_int32),
        ("heads", C.c_int32), ("head_mean", C.c_int32), ("neg_slope", C.c_float), ("act", C.c_int),
        ("edge_feat", C.c_int32),
        ("w", C.c_void_p), ("b", C.c_void_p), ("w_pool", C.c_void_p), ("b_pool", C.c_void_p),
        ("attn_l", C.c_void_p), ("attn_r", C.c_void_p), ("w_e", C.c_void_p), ("b_e", C.c_void_p),
        ("w_ih", C.c_void_p), ("b_ih", C.c_void_p), ("w_hh", C.c_void_p), ("b_hh", C.c_void_p),
        ("hidden", C.c_int32), ("w_self", C.c_void_p), ("rel", C.POINTER(saga_rel_plan)),
    ]


_lib = None


def lib():
    """Load libsaga.so (raises if it is missing: there is no fallback)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} not built; run paper_2009_00804_amd.build.build()")
    L = C.CDLL(LIB_PATH)
    P = C.POINTER
    S = C.c_int
    sig = {
        "saga_plan_workspace_size": (S, [C.c_int32, C.c_int32, C.c_int64, P(saga_plan_opts), P(C.c_size_t)]),
        "saga_plan_build": (S, [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_void_p, P(saga_plan_opts),
                                C.c_void_p, C.c_size_t, C.c_void_p, P(saga_plan)]),
        "saga_plan_build_split": (S, [C.c_int32, C.c_int32, C.c_int64, C.c_void_p, C.c_void_p,
                                      P(saga_plan_opts), C.c_void_p, C.c_size_t, C.c_void_p,
                                      C.c_void_p, C.c_void_p, C.c_void_p, P(saga_plan)]),
        "saga_plan_check": (S, [P(saga_plan), C.c_void_p, P(saga_plan_counts)]),
        "saga_gather_workspace_size": (S, [P(saga_plan), P(saga_edge_op), C.c_int64, P(C.c_size_t)]),
        "saga_scatter_apply_edge_gather": (S, [P(saga_plan), P(saga_edge_op), P(saga_edge_inputs), saga_mat,
                                               C.c_void_p, C.c_size_t, C.c_void_p]),
        "saga_scatter_apply_edge_gather_noalloc": (S, [P(saga_plan), P(saga_edge_op), P(saga_edge_inputs),
                                                       saga_mat, C.c_void_p]),
        "saga_gather_transform_workspace_size": (S, [P(saga_plan), P(saga_edge_op), C.c_int64,
                                                     P(C.c_size_t)]),
        "saga_scatter_apply_edge_gather_transform": (S, [P(saga_plan), P(saga_edge_op), P(saga_edge_inputs),
                                                         P(saga_next_transform), saga_mat, C.c_void_p,
                                                         C.c_size_t, C.c_void_p]),
        "saga_unfused_workspace_size": (S, [P(saga_plan), P(saga_edge_op), C.c_int64, P(C.c_size_t)]),
        "saga_scatter_gather_unfused": (S, [P(saga_plan), P(saga_edge_op), P(saga_edge_inputs), saga_mat,
                                            C.c_void_p, C.c_size_t, C.c_void_p]),
        "saga_lstm_gather_workspace_size": (S, [P(saga_plan), C.c_int64, P(C.c_size_t)]),
        "saga_lstm_gather": (S, [P(saga_plan), saga_cmat, saga_cmat, saga_mat, C.c_void_p, C.c_size_t,
                                 C.c_void_p]),
        "saga_lstm_gather_rows": (S, [P(saga_plan), C.c_int32, C.c_int32, saga_cmat, saga_cmat,
                                      saga_mat, C.c_void_p, C.c_size_t, C.c_void_p]),
        "saga_rel_plan_workspace_size": (S, [P(saga_plan), C.c_int32, P(C.c_size_t)]),
        "saga_rel_plan_build": (S, [P(saga_plan), C.c_void_p, C.c_int32, C.c_void_p, C.c_size_t,
                                    C.c_void_p, P(saga_rel_plan)]),
        "saga_rel_plan_check": (S, [P(saga_rel_plan), C.c_void_p, P(saga_rel_counts)]),
        "saga_rel_transform_workspace_size": (S, [P(saga_rel_plan), C.c_int, C.c_int64, C.c_int64,
                                                  P(C.c_size_t)]),
        "saga_rel_transform": (S, [P(saga_rel_plan), C.c_int, saga_cmat, saga_cmat, saga_mat,
                                   C.c_void_p, C.c_size_t, C.c_void_p]),
        "saga_apply_vertex_workspace_size": (S, [P(saga_gemm_op), C.c_int64, C.c_int64, C.c_int64,
                                                 P(C.c_size_t)]),
        "saga_apply_vertex": (S, [P(saga_gemm_op), saga_cmat, saga_cmat, saga_cmat, saga_cmat, C.c_void_p,
                                  C.c_void_p, saga_mat, C.c_void_p, C.c_size_t, C.c_void_p]),
        "saga_layer_workspace_size": (S, [P(saga_plan), P(saga_layer_desc), P(C.c_size_t)]),
        "saga_layer": (S, [P(saga_plan), P(saga_layer_desc), saga_cmat, saga_cmat, saga_mat, C.c_void_p,
                           C.c_size_t, C.c_void_p]),
        "saga_trace_stages": (S, [C.POINTER(C.c_void_p), C.c_int32, C.c_int32]),
        "saga_sync_check": (S, [C.c_void_p]),
        "saga_status_str": (C.c_char_p, [S]),
        "saga_last_error": (C.c_char_p, []),
        "saga_version": (C.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        f = getattr(L, name)
        f.restype = res
        f.argtypes = args
    _lib = L
    return L


class SagaError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        detail = lib().saga_last_error().decode()
        name = lib().saga_status_str(status).decode()
        super().__init__(f"{where}: {name} ({status}): {detail}")


def _check(status, where):
    if status != SAGA_OK:
        raise SagaError(status, where)
    return status


# --------------------------------------------------------------------------
# the C entry points, same names
# --------------------------------------------------------------------------
def saga_plan_workspace_size(num_dst, num_src, num_edges, opts=None):
    out = C.c_size_t(0)
    _check(lib().saga_plan_workspace_size(num_dst, num_src, num_edges,
                                          C.byref(opts) if opts else None, C.byref(out)),
           "saga_plan_workspace_size")
    return out.value


def saga_plan_build(num_dst, num_src, num_edges, row_ptr, col_idx, opts, workspace, ws_bytes, stream):
    plan = saga_plan()
    _check(lib().saga_plan_build(num_dst, num_src, num_edges, row_ptr, col_idx,
                                 C.byref(opts) if opts else None, workspace, ws_bytes, stream,
                                 C.byref(plan)), "saga_plan_build")
    return plan


def saga_plan_build_split(num_dst, num_src, num_edges, row_ptr, col_idx, opts, workspace, ws_bytes,
                          stream, order_stream, fork_event, join_event):
    plan = saga_plan()
    _check(lib().saga_plan_build_split(num_dst, num_src, num_edges, row_ptr, col_idx,
                                       C.byref(opts) if opts else None, workspace, ws_bytes, stream,
                                       order_stream, fork_event, join_event, C.byref(plan)),
           "saga_plan_build_split")
    return plan


def saga_plan_check(plan, stream):
    counts = saga_plan_counts()
    st = lib().saga_plan_check(C.byref(plan), stream, C.byref(counts))
    return st, counts


def saga_gather_workspace_size(plan, op, feat):
    out = C.c_size_t(0)
    _check(lib().saga_gather_workspace_size(C.byref(plan), C.byref(op), feat, C.byref(out)),
           "saga_gather_workspace_size")
    return out.value


def saga_scatter_apply_edge_gather(plan, op, inputs, out, workspace, ws_bytes, stream):
    return _check(lib().saga_scatter_apply_edge_gather(C.byref(plan), C.byref(op), C.byref(inputs), out,
                                                       workspace, ws_bytes, stream),
                  "saga_scatter_apply_edge_gather")


def saga_scatter_apply_edge_gather_noalloc(plan, op, inputs, out, stream):
    return _check(lib().saga_scatter_apply_edge_gather_noalloc(C.byref(plan), C.byref(op), C.byref(inputs),
                                                               out, stream),
                  "saga_scatter_apply_edge_gather_noalloc")


def saga_gather_transform_workspace_size(plan, op, feat):
    out = C.c_size_t(0)
    _check(lib().saga_gather_transform_workspace_size(C.byref(plan), C.byref(op), feat, C.byref(out)),
           "saga_gather_transform_workspace_size")
    return out.value


def saga_scatter_apply_edge_gather_transform(plan, op, inputs, nxt, out, workspace, ws_bytes, stream):
    return _check(lib().saga_scatter_apply_edge_gather_transform(
        C.byref(plan), C.byref(op), C.byref(inputs), C.byref(nxt), out, workspace, ws_bytes, stream),
        "saga_scatter_apply_edge_gather_transform")


def saga_unfused_workspace_size(plan, op, feat):
    out = C.c_size_t(0)
    _check(lib().saga_unfused_workspace_size(C.byref(plan), C.byref(op), feat, C.byref(out)),
           "saga_unfused_workspace_size")
    return out.value


def saga_scatter_gather_unfused(plan, op, inputs, out, workspace, ws_bytes, stream):
    return _check(lib().saga_scatter_gather_unfused(C.byref(plan), C.byref(op), C.byref(inputs), out,
                                                    workspace, ws_bytes, stream),
                  "saga_scatter_gather_unfused")


def saga_lstm_gather_workspace_size(plan, hidden):
    out = C.c_size_t(0)
    _check(lib().saga_lstm_gather_workspace_size(C.byref(plan), hidden, C.byref(out)),
           "saga_lstm_gather_workspace_size")
    return out.value


def saga_lstm_gather(plan, gates_x, w_hh, out, workspace, ws_bytes, stream):
    return _check(lib().saga_lstm_gather(C.byref(plan), gates_x, w_hh, out, workspace, ws_bytes, stream),
                  "saga_lstm_gather")


def saga_rel_plan_workspace_size(plan, num_rel):
    out = C.c_size_t(0)
    _check(lib().saga_rel_plan_workspace_size(C.byref(plan), num_rel, C.byref(out)),
           "saga_rel_plan_workspace_size")
    return out.value


def saga_rel_plan_build(plan, etype, num_rel, workspace, ws_bytes, stream):
    rel = saga_rel_plan()
    _check(lib().saga_rel_plan_build(C.byref(plan), etype, num_rel, workspace, ws_bytes, stream,
                                     C.byref(rel)), "saga_rel_plan_build")
    return rel


def saga_rel_plan_check(rel, stream):
    counts = saga_rel_counts()
    st = lib().saga_rel_plan_check(C.byref(rel), stream, C.byref(counts))
    return st, counts


def saga_rel_transform_workspace_size(rel, dtype, k, n):
    out = C.c_size_t(0)
    _check(lib().saga_rel_transform_workspace_size(C.byref(rel), dtype, k, n, C.byref(out)),
           "saga_rel_transform_workspace_size")
    return out.value


def saga_rel_transform(rel, dtype, x, w, out, workspace, ws_bytes, stream):
    return _check(lib().saga_rel_transform(C.byref(rel), dtype, x, w, out, workspace, ws_bytes,
                                           stream), "saga_rel_transform")


def saga_lstm_gather_rows(plan, perm_begin, perm_end, gates_x, w_hh, out, workspace, ws_bytes,
                          stream):
    return _check(lib().saga_lstm_gather_rows(C.byref(plan), perm_begin, perm_end, gates_x, w_hh, out,
                                              workspace, ws_bytes, stream),
                  "saga_lstm_gather_rows")


def saga_apply_vertex_workspace_size(op, k, k2, n):
    out = C.c_size_t(0)
    _check(lib().saga_apply_vertex_workspace_size(C.byref(op), k, k2, n, C.byref(out)),
           "saga_apply_vertex_workspace_size")
    return out.value


def saga_apply_vertex(op, a, w, a2, w2, bias, bias2, out, workspace, ws_bytes, stream):
    return _check(lib().saga_apply_vertex(C.byref(op), a, w, a2, w2, bias, bias2, out, workspace,
                                          ws_bytes, stream),
                  "saga_apply_vertex")


def saga_trace_stages(events, markers=False):
    """Record events[i] (torch.cuda.Event) after stage i of each saga_layer
    call on this thread; saga_trace_stages([]) stops."""
    for e in events:
        if not e.cuda_event:      # torch creates the event at its first record
            e.record()
    handles = [e.cuda_event for e in events]
    arr = (C.c_void_p * max(1, len(handles)))(*handles)
    return _check(lib().saga_trace_stages(arr if handles else None, len(handles), int(markers)),
                  "saga_trace_stages")


def saga_layer_workspace_size(plan, desc):
    out = C.c_size_t(0)
    _check(lib().saga_layer_workspace_size(C.byref(plan), C.byref(desc), C.byref(out)),
           "saga_layer_workspace_size")
    return out.value


def saga_layer(plan, desc, x, edge_feat, out, workspace, ws_bytes, stream):
    return _check(lib().saga_layer(C.byref(plan), C.byref(desc), x, edge_feat, out, workspace,
                                   ws_bytes, stream), "saga_layer")


def saga_version():
    return lib().saga_version().decode()


def saga_sync_check(stream):
    return _check(lib().saga_sync_check(stream), "saga_sync_check")


# --------------------------------------------------------------------------
# torch marshalling helpers
# --------------------------------------------------------------------------
def dtype_code(t: torch.dtype) -> int:
    if t == torch.float32:
        return SAGA_F32
    if t == torch.bfloat16:
        return SAGA_BF16
    raise ValueError(f"unsupported dtype {t}")


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def cmat(t, rows=None, cols=None):
    """saga_cmat view of a 2-D tensor (row-major with unit column stride)."""
    if t is None:
        return saga_cmat(None, 0, 0, 0)
    assert t.dim() == 2 and t.stride(1) == 1, "matrix must be row-major with unit column stride"
    return saga_cmat(t.data_ptr(), rows if rows is not None else t.shape[0],
                     cols if cols is not None else t.shape[1], t.stride(0))


def mat(t, rows=None, cols=None):
    assert t.dim() == 2 and t.stride(1) == 1
    return saga_mat(t.data_ptr(), rows if rows is not None else t.shape[0],
                    cols if cols is not None else t.shape[1], t.stride(0))


def gather_ld(cols, elem_size):
    """Leading dimension (elements) for a matrix whose rows the gather
    fetches: rows up to 128 bytes padded to a power of two, longer rows to a
    multiple of 64 bytes, so a row never touches more 128-byte L2 lines than
    it must (the rule saga_layer uses for its intermediates)."""
    b = cols * elem_size
    if b <= 128:
        p = 16
        while p < b:
            p <<= 1
        b = p
    else:
        b = (b + 63) // 64 * 64
    return b // elem_size


def padded_empty(rows, cols, dtype, device, align_elems=None):
    """rows x cols view of a buffer whose rows are padded to 16 bytes."""
    es = torch.tensor([], dtype=dtype).element_size()
    a = align_elems or (16 // es)
    ld = (cols + a - 1) // a * a
    buf = torch.empty((rows, ld), dtype=dtype, device=device)
    return buf[:, :cols]


def stream_handle(stream=None):
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def workspace(nbytes, device):
    n = max(256, (int(nbytes) + 255) // 256 * 256)
    return torch.empty(n, dtype=torch.uint8, device=device)


class Graph:
    """A device-resident in-CSR and its plan (all memory owned by torch)."""

    def __init__(self, row_ptr, col_idx, num_src=None, seg_len=0, block_cost=0, row_cost=0,
                 stream=None, check=True):
        assert row_ptr.dtype == torch.int32 and col_idx.dtype == torch.int32
        self.row_ptr = row_ptr
        self.col_idx = col_idx
        self.num_dst = row_ptr.numel() - 1
        self.num_src = self.num_dst if num_src is None else num_src
        self.num_edges = col_idx.numel()
        self.opts = saga_plan_opts(seg_len, block_cost, row_cost)
        self.ws_bytes = saga_plan_workspace_size(self.num_dst, self.num_src, self.num_edges, self.opts)
        self.ws = workspace(self.ws_bytes, row_ptr.device)
        self.stream = stream
        self.build()
        self.counts = None
        if check:
            self.check()

    def build(self):
        self.plan = saga_plan_build(self.num_dst, self.num_src, self.num_edges, _ptr(self.row_ptr),
                                    _ptr(self.col_idx) if self.num_edges else None, self.opts,
                                    _ptr(self.ws), self.ws.numel(), stream_handle(self.stream))
        return self.plan

    def check(self):
        st, counts = saga_plan_check(self.plan, stream_handle(self.stream))
        self.counts = counts
        _check(st, "saga_plan_check")
        return counts

    def _view(self, ptr, n):
        """int32 tensor view of n ints of the plan workspace at device address ptr."""
        if n == 0:
            return torch.zeros(0, dtype=torch.int32, device=self.ws.device)
        off = ptr - self.ws.data_ptr()
        return self.ws[off:off + 4 * n].view(torch.int32)

    def arrays(self):
        """Plan arrays as int32 tensors (views into the workspace)."""
        c = self.counts or self.check()
        p = self.plan
        V, S, nb = self.num_dst, c.num_segments, c.num_blocks
        return dict(
            d_in=self._view(p.d_in, V), d_out=self._view(p.d_out, self.num_src),
            perm=self._view(p.perm, V), row_seg_first=self._view(p.row_seg_first, V + 1),
            seg_row=self._view(p.seg_row, S), seg_beg=self._view(p.seg_beg, S),
            seg_end=self._view(p.seg_end, S), block_ptr=self._view(p.block_ptr, nb + 1))


class RelGraph:
    """The typed layout of a Graph's edges (R-GCN): etype is an int32 device
    tensor aligned with the CSR entries; memory owned by torch."""

    def __init__(self, graph: Graph, etype, num_rel, stream=None, check=True):
        assert etype.dtype == torch.int32 and etype.numel() == graph.num_edges
        self.graph = graph
        self.etype = etype
        self.num_rel = num_rel
        self.stream = stream
        self.ws_bytes = saga_rel_plan_workspace_size(graph.plan, num_rel)
        self.ws = workspace(self.ws_bytes, etype.device)
        self.build()
        self.counts = None
        if check:
            self.check()

    def build(self):
        self.rel = saga_rel_plan_build(self.graph.plan, _ptr(self.etype) if self.etype.numel() else None,
                                       self.num_rel, _ptr(self.ws), self.ws.numel(),
                                       stream_handle(self.stream))
        return self.rel

    def check(self):
        st, counts = saga_rel_plan_check(self.rel, stream_handle(self.stream))
        self.counts = counts
        _check(st, "saga_rel_plan_check")
        return counts

    def _view(self, ptr, n, dtype=torch.int32):
        if n == 0:
            return torch.zeros(0, dtype=dtype, device=self.ws.device)
        off = ptr - self.ws.data_ptr()
        return self.ws[off:off + 4 * n].view(dtype)

    def arrays(self):
        c = self.counts or self.check()
        r = self.rel
        E = self.graph.num_edges
        return dict(rel_ptr=self._view(r.rel_ptr, self.num_rel + 1),
                    rel_count=self._view(r.rel_count, self.num_rel),
                    pair_src=self._view(r.pair_src, c.pair_rows),
                    edge_pair=self._view(r.edge_pair, E),
                    edge_norm=self._view(r.edge_norm, E, torch.float32))
