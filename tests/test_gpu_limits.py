"""The largest CSR a plan accepts: with 2^21 vertices, seg_len 512 and
row_cost 4 that is 2,122,512,902 edges (the total segment cost just below
2^31; every int32 edge offset in use up to there), with one hub row of
4.4 M in-edges and every other row of 1010.

col_idx[e] = e mod V for every CSR entry e, so the results have closed
forms that need no per-edge oracle pass over two billion edges: d_out[u] =
E div V (+1 for u < E mod V), the degree order is the hub then every other
row in id order, the sum of ones over a row is its in-degree, and the max of
the source ids over a row is the last id of its run of consecutive ids
(V - 1 if the run wraps).  The segment table and row blocks come from the
oracle's own (per-row) definitions."""
import ctypes as C

import numpy as np
import pytest
import torch

from gpu_util import device, lib
from helpers import plan_edge_limit
from oracle import saga_oracle as O

pytestmark = [pytest.mark.gpu, pytest.mark.slow]

V = 1 << 21
SEG_LEN, BLOCK_COST, ROW_COST = 512, 4096, 4
E = plan_edge_limit(V, SEG_LEN, ROW_COST)
D = 1010                   # in-degree of every row but the hub (row 0)


@pytest.fixture(scope="module")
def limit_graph():
    S = lib()
    dev = device()
    d_in = np.full(V, D, np.int64)
    d_in[0] = E - D * (V - 1)
    rp = np.zeros(V + 1, np.int64)
    np.cumsum(d_in, out=rp[1:])
    assert rp[-1] == E and d_in[0] > D and d_in[0] < 2**24
    print(f"limit graph: V={V} E={E} hub in-degree {d_in[0]}", flush=True)
    row_ptr = torch.from_numpy(rp.astype(np.int32)).to(dev)
    col = torch.empty(E, dtype=torch.int32, device=dev)
    step = 1 << 28
    for e0 in range(0, E, step):  # e mod V, built in pieces on the device
        e1 = min(E, e0 + step)
        col[e0:e1] = (torch.arange(e0, e1, dtype=torch.int64, device=dev) % V).to(torch.int32)
    torch.cuda.synchronize()
    g = S.Graph(row_ptr, col, seg_len=SEG_LEN, block_cost=BLOCK_COST, row_cost=ROW_COST)
    return g, rp, d_in


def test_limit_plan(limit_graph):
    g, rp, d_in = limit_graph
    a = {k: v.cpu().numpy().astype(np.int64) for k, v in g.arrays().items()}
    assert np.array_equal(a["d_in"], d_in)
    want_out = np.full(V, E // V, np.int64)
    want_out[: E % V] += 1
    assert np.array_equal(a["d_out"], want_out)
    perm = np.arange(V)  # the hub first, then the equal degrees by id
    assert np.array_equal(a["perm"], perm)
    assert np.array_equal(perm, O.degree_order(d_in))
    # segments and row blocks: the oracle's definitions (vectorised; the
    # only per-edge work of the oracle plan is the out-degree count, whose
    # closed form is used above)
    p = g.plan
    seg_row, seg_beg, seg_end, first = O.segments(rp, perm, p.seg_len)
    assert np.array_equal(a["row_seg_first"], first)
    assert np.array_equal(a["seg_row"], seg_row)
    assert np.array_equal(a["seg_beg"], seg_beg)
    assert np.array_equal(a["seg_end"], seg_end)
    assert np.array_equal(a["block_ptr"], O.row_blocks(seg_beg, seg_end, p.block_cost, p.row_cost))
    assert g.counts.n_split == int(np.count_nonzero(np.diff(first) > 1))
    assert int((seg_end - seg_beg).sum()) == E


def _gather(g, src, reduce):
    S = lib()
    op = S.saga_edge_op()
    op.msg = S.SAGA_MSG_COPY
    op.reduce = reduce
    op.dtype = S.dtype_code(src.dtype)
    op.heads = 1
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(src)
    out = torch.full((V, 4), 7.0, dtype=torch.float32, device=src.device)[:, :1]
    n = S.saga_gather_workspace_size(g.plan, op, 1)
    ws = S.workspace(n, src.device)
    S.saga_scatter_apply_edge_gather(g.plan, op, inp, S.mat(out), C.c_void_p(ws.data_ptr()),
                                     ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    return out[:, 0].cpu().numpy().astype(np.float64)


def test_limit_gather_sum_and_max(limit_graph):
    g, rp, d_in = limit_graph
    S = lib()
    dev = device()
    ones = torch.ones((V, 4), dtype=torch.float32, device=dev)[:, :1]
    print("limit gather: sum of ones", flush=True)
    got = _gather(g, ones, S.SAGA_RED_SUM)
    assert np.array_equal(got, d_in.astype(np.float64))  # exact: in-degrees < 2^24
    ids = torch.arange(V, dtype=torch.float32, device=dev).view(V, 1).expand(V, 4).contiguous()
    print("limit gather: max of source ids", flush=True)
    got = _gather(g, ids[:, :1], S.SAGA_RED_MAX)
    e0, e1 = rp[:-1], rp[1:] - 1
    s0, s1 = e0 % V, e1 % V
    want = np.where((e1 - e0 + 1 >= V) | (s0 > s1), V - 1, s1).astype(np.float64)
    assert np.array_equal(got, want)
