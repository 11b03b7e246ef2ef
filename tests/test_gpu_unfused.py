"""Parity of the unfused baseline (Sec. 3.2 "Gather", Fig. 7a: a
materialised edge tensor, then a segment reduction) against the CPU oracle
and against the fused kernel, on the op-level graphs of test_gpu_ops plus an
edgeless graph."""
import ctypes as C

import numpy as np
import pytest
import torch

from gpu_util import dev_padded, device, graph, lib, to_np
from helpers import BF16_TOL, FP32_TOL, edges_to_csr, rel_err
from oracle import saga_oracle as O
from test_gpu_ops import ACTS, _bf16_round, _get_graph, _ref_simple, run_gather

pytestmark = pytest.mark.gpu


def run_unfused(g, src_t, op_kw, out_cols, out_dtype, bias=None):
    S = lib()
    op = S.saga_edge_op()
    op.msg = op_kw.get("msg", S.SAGA_MSG_COPY)
    op.reduce = op_kw["reduce"]
    op.dtype = S.dtype_code(src_t.dtype)
    op.heads = 1
    op.dst_norm = op_kw.get("dst_norm", 0)
    op.act = ACTS[op_kw.get("act", "none")]
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(src_t)
    bias_t = None
    if bias is not None:
        bias_t = torch.from_numpy(np.asarray(bias, np.float32)).to(device())
        inp.bias = bias_t.data_ptr()
    out = dev_padded(np.zeros((g.num_dst, out_cols)), dtype=out_dtype, fill=7.0)
    n = S.saga_unfused_workspace_size(g.plan, op, src_t.shape[1])
    ws = S.workspace(n, device())
    S.saga_scatter_gather_unfused(g.plan, op, inp, S.mat(out), C.c_void_p(ws.data_ptr()),
                                  ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("gname", ["rmat", "tiny_multi", "tiny_star", "tiny_random", "tiny_chain"])
@pytest.mark.parametrize("F", [1, 8, 41, 128, 300, 602])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_unfused_matches_oracle(gname, F, dtype):
    S = lib()
    rp, col, n, g = _get_graph(gname)
    rng = np.random.default_rng(1000 + F)
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
        print(f"unfused {gname} F={F} {dtype} {red} {msg} dst_norm={dn} act={act}", flush=True)
        out = run_unfused(g, Xt, dict(reduce={"sum": S.SAGA_RED_SUM, "mean": S.SAGA_RED_MEAN}[red],
                                      msg={"copy": S.SAGA_MSG_COPY, "src_norm": S.SAGA_MSG_SRC_NORM}[msg],
                                      dst_norm=dn, act=act), F, tdt, bias=b)
        ref = _ref_simple(rp, col, X, red, msg, dn, b, act, n)
        assert rel_err(to_np(out), ref) <= tol, (red, msg)
    print(f"unfused {gname} F={F} {dtype} max", flush=True)
    out = run_unfused(g, Xt, dict(reduce=S.SAGA_RED_MAX), F, tdt)
    assert np.array_equal(to_np(out), O.gather(rp, col, X, "max"))


@pytest.mark.parametrize("F", [16, 128])
def test_unfused_equals_fused_where_order_free(F):
    """MAX is order-independent and float32 COPY messages are not rounded,
    so the unfused max equals the fused max bit for bit."""
    S = lib()
    rp, col, n, g = _get_graph("rmat")
    X = np.random.default_rng(F).standard_normal((n, F)).astype(np.float32)
    Xt = dev_padded(X)
    for msg in (S.SAGA_MSG_COPY, S.SAGA_MSG_SRC_NORM):
        print(f"unfused vs fused max F={F} msg={msg}", flush=True)
        a = run_unfused(g, Xt, dict(reduce=S.SAGA_RED_MAX, msg=msg), F, torch.float32)
        b = run_gather(g, Xt, dict(reduce=S.SAGA_RED_MAX, msg=msg), F, torch.float32)
        assert torch.equal(a.cpu(), b.cpu())


def test_unfused_edgeless_graph():
    S = lib()
    n = 37
    rp = np.zeros(n + 1, np.int32)
    col = np.zeros(0, np.int32)
    g = graph(rp, col, num_src=n)
    X = np.random.default_rng(3).standard_normal((n, 24)).astype(np.float32)
    bias = np.linspace(-1, 1, 24)
    print("unfused edgeless", flush=True)
    out = run_unfused(g, dev_padded(X), dict(reduce=S.SAGA_RED_SUM, act="relu"), 24, torch.float32,
                      bias=bias)
    assert np.array_equal(to_np(out), np.broadcast_to(np.maximum(bias, 0).astype(np.float32), (n, 24)))


def test_unfused_deterministic():
    S = lib()
    rp, col, n, g = _get_graph("rmat")
    X = np.random.default_rng(9).standard_normal((n, 128)).astype(np.float32)
    Xt = dev_padded(X)
    a = run_unfused(g, Xt, dict(reduce=S.SAGA_RED_SUM, dst_norm=1), 128, torch.float32)
    b = run_unfused(g, Xt, dict(reduce=S.SAGA_RED_SUM, dst_norm=1), 128, torch.float32)
    assert torch.equal(a.cpu(), b.cpu())
