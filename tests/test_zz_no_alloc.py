"""The allocation-free Gather (saga_scatter_apply_edge_gather_noalloc)
against the workspace Gather it is a variant of: two calls in a row on the
same fixed device scratch, the second on a smaller graph, each compared
with saga_scatter_apply_edge_gather bit for bit; and the size limit
refused on the host before anything runs."""
import ctypes as C

import numpy as np
import pytest
import torch

from gpu_util import dev_padded, device, graph, lib
from helpers import edges_to_csr

pytestmark = pytest.mark.gpu


def _rmat_graph(scale, deg, key):
    from synth import graphs as G
    from synth.configs import RMAT_ABC

    n = 1 << scale
    src, dst = G.rmat(scale, deg * n, *RMAT_ABC, key=(key, 0))
    res = G.to_in_csr(n, src, dst)
    return res[0], res[1], n


def _op(S, reduce, dtype, dst_norm, act):
    op = S.saga_edge_op()
    op.msg = S.SAGA_MSG_COPY
    op.reduce = reduce
    op.dtype = dtype
    op.heads = 1
    op.dst_norm = dst_norm
    op.act = act
    return op


def _both(S, g, op, src_t, bias):
    """Outputs of the workspace Gather and of the allocation-free one."""
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(src_t)
    bias_t = None
    if bias is not None:
        bias_t = torch.from_numpy(np.asarray(bias, np.float32)).to(device())
        inp.bias = bias_t.data_ptr()
    F = src_t.shape[1]
    want = dev_padded(np.zeros((g.num_dst, F)), dtype=src_t.dtype, fill=7.0)
    got = dev_padded(np.zeros((g.num_dst, F)), dtype=src_t.dtype, fill=-3.0)
    ws = S.workspace(S.saga_gather_workspace_size(g.plan, op, F), device())
    S.saga_scatter_apply_edge_gather(g.plan, op, inp, S.mat(want), C.c_void_p(ws.data_ptr()),
                                     ws.numel(), S.stream_handle())
    S.saga_scatter_apply_edge_gather_noalloc(g.plan, op, inp, S.mat(got), S.stream_handle())
    torch.cuda.synchronize()
    return want, got


def test_noalloc_gather_equals_workspace_gather_twice():
    S = lib()
    rng = np.random.default_rng(31)
    # call 1: 2^14-vertex power-law graph, hub rows split into segments
    # (partials in the fixed scratch), float32, sum with d_in^-1/2, bias, ReLU
    rp, col, n = _rmat_graph(14, 16, 131)
    g = graph(rp, col)
    c = g.check()
    assert c.n_split > 0, "the first graph must have split rows"
    print(f"noalloc call 1: V={n} E={len(col)} split rows {c.n_split}", flush=True)
    X = dev_padded(rng.standard_normal((n, 128)))
    op = _op(S, S.SAGA_RED_SUM, S.SAGA_F32, 1, S.SAGA_ACT_RELU)
    want, got = _both(S, g, op, X, rng.standard_normal(128))
    assert torch.equal(got, want)
    # call 2, smaller: 2^11-vertex graph, bfloat16, mean, no bias; the
    # scratch still holds call 1's partials
    rp2, col2, n2 = _rmat_graph(11, 24, 132)
    g2 = graph(rp2, col2)
    c2 = g2.check()
    assert c2.n_split > 0 and n2 < n
    print(f"noalloc call 2: V={n2} E={len(col2)} split rows {c2.n_split}", flush=True)
    X2 = dev_padded(rng.standard_normal((n2, 64)), dtype=torch.bfloat16)
    op2 = _op(S, S.SAGA_RED_MEAN, S.SAGA_BF16, 0, S.SAGA_ACT_NONE)
    want2, got2 = _both(S, g2, op2, X2, None)
    assert torch.equal(got2, want2)


def test_noalloc_gather_refuses_partials_beyond_its_scratch():
    S = lib()
    # segments of one edge: the host bound on split-row partials is
    # (E + min(E / 2, V)) segments x 128 floats = 150,000 x 512 B = 76.8 MB,
    # above the 64 MiB scratch: refused before any launch
    n = 50000
    src = np.arange(100000) % n
    dst = (np.arange(100000) * 7) % n
    rp, col, _ = edges_to_csr(n, src.tolist(), dst.tolist())
    g = graph(rp, col, seg_len=1, block_cost=8, row_cost=1)
    op = _op(S, S.SAGA_RED_SUM, S.SAGA_F32, 0, S.SAGA_ACT_NONE)
    X = dev_padded(np.ones((n, 128)))
    out = dev_padded(np.full((n, 128), 5.0))
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(X)
    with pytest.raises(S.SagaError) as ei:
        S.saga_scatter_apply_edge_gather_noalloc(g.plan, op, inp, S.mat(out), S.stream_handle())
    assert ei.value.status == S.SAGA_EUNSUPPORTED
    assert "fixed scratch" in str(ei.value)
    torch.cuda.synchronize()
    assert bool(torch.all(out == 5.0))
