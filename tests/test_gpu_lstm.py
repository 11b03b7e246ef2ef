"""Parity of the LSTM Gather (GraphSAGE row of Table I) and of the
GraphSAGE-LSTM layer against the oracle: tiny graphs, a power-law graph
whose longest row crosses the kernel's neighbour-id chunk boundary, a row of
several thousand in-edges, empty rows, and H = 32, 64, 128."""
import ctypes as C

import numpy as np
import pytest
import torch

from gpu_util import dev_padded, device, graph, lib, to_np
from helpers import FP32_TOL, edges_to_csr, rel_err, tiny_graphs
from oracle import saga_oracle as O

pytestmark = pytest.mark.gpu


def run_lstm(g, P, W_hh):
    S = lib()
    H = W_hh.shape[0]
    Pt = dev_padded(P)
    Wt = torch.from_numpy(np.ascontiguousarray(W_hh, np.float32)).to(device())
    out = dev_padded(np.zeros((g.num_dst, H)), fill=5.0)
    ws = S.workspace(S.saga_lstm_gather_workspace_size(g.plan, H), device())
    S.saga_lstm_gather(g.plan, S.cmat(Pt), S.cmat(Wt), S.mat(out), C.c_void_p(ws.data_ptr()),
                       ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    return to_np(out)


def _ref(rp, col, P, W_hh):
    """The oracle's LSTM Gather fed the input part of the gates directly
    (x = P, W_ih = identity, zero biases)."""
    G = P.shape[1]
    z = np.zeros(G)
    return O.lstm_gather(rp, col, P.astype(np.float64), np.eye(G), z, W_hh.astype(np.float64), z)


def _graphs():
    out = []
    for name, n, src, dst in tiny_graphs():
        rp, col, _ = edges_to_csr(n, src, dst)
        out.append((name, n, rp, col))
    from synth import configs as Cfg

    g = Cfg.build("sage_lstm", small=True)       # longest row: 1035 in-edges
    out.append(("rmat", g["num_vertices"], g["row_ptr"], g["col_idx"]))
    # one row of 3000 in-edges (three id chunks), short rows, empty rows
    rng = np.random.default_rng(4)
    n = 200
    d = np.zeros(n, np.int64)
    d[7], d[8], d[9] = 3000, 1, 13
    d[20:60] = rng.integers(1, 40, 40)
    rp = np.concatenate([[0], np.cumsum(d)]).astype(np.int32)
    col = rng.integers(0, n, int(rp[-1])).astype(np.int32)
    out.append(("long_row", n, rp, col))
    return out


@pytest.mark.parametrize("case", _graphs(), ids=lambda c: c[0])
@pytest.mark.parametrize("H", [32, 64, 128])
def test_lstm_gather_matches_oracle(case, H):
    name, n, rp, col = case
    rng = np.random.default_rng(H)
    P = rng.standard_normal((n, 4 * H)).astype(np.float32)
    a = 1.0 / np.sqrt(H)
    W_hh = rng.uniform(-a, a, (H, 4 * H)).astype(np.float32)
    print(f"lstm gather {name} H={H}", flush=True)
    g = graph(rp, col, num_src=n)
    got = run_lstm(g, P, W_hh)
    want = _ref(rp, col, P, W_hh)
    assert rel_err(got, want) <= FP32_TOL
    assert np.array_equal(got[np.diff(rp) == 0], np.zeros(((np.diff(rp) == 0).sum(), H), np.float32))


def test_lstm_gather_deterministic_and_repeatable():
    name, n, rp, col = _graphs()[-2]
    H = 128
    rng = np.random.default_rng(1)
    P = rng.standard_normal((n, 4 * H)).astype(np.float32)
    W_hh = rng.uniform(-0.09, 0.09, (H, 4 * H)).astype(np.float32)
    g = graph(rp, col, num_src=n)
    print("lstm gather repeat", flush=True)
    a = run_lstm(g, P, W_hh)
    b = run_lstm(g, P, W_hh)
    assert np.array_equal(a, b)


def test_sage_lstm_layer():
    from paper_2009_00804_amd import layers as LY
    from synth import configs as Cfg

    g = Cfg.build("sage_lstm", small=True)
    S = lib()
    gr = S.Graph(torch.from_numpy(g["row_ptr"]).to(device()), torch.from_numpy(g["col_idx"]).to(device()))
    print("sage-lstm layer", flush=True)
    y = to_np(LY.run(LY.sage_lstm(gr, g), dev_padded(g["X"])))
    want = O.sage_lstm_layer_of(g)
    assert rel_err(y, want) <= FP32_TOL


def test_lstm_rows_degree_traversal_equals_single_call():
    """One saga_lstm_gather_rows call per run of equal in-degree (the degree
    traversal of Sec. 3.2) writes the same bytes as the single call; a
    partial range writes only its own rows."""
    S = lib()
    name, n, rp, col = _graphs()[-2]
    H = 64
    rng = np.random.default_rng(11)
    P = rng.standard_normal((n, 4 * H)).astype(np.float32)
    W_hh = rng.uniform(-0.12, 0.12, (H, 4 * H)).astype(np.float32)
    g = graph(rp, col, num_src=n)
    print("lstm degree traversal", flush=True)
    full = run_lstm(g, P, W_hh)
    arr = g.arrays()
    perm = arr["perm"].cpu().numpy()
    dsorted = arr["d_in"].cpu().numpy()[perm]
    cuts = np.concatenate([[0], np.flatnonzero(np.diff(dsorted)) + 1, [n]])
    Pt = dev_padded(P)
    Wt = torch.from_numpy(W_hh).to(device())
    out = dev_padded(np.zeros((n, H)), fill=5.0)
    ws = S.workspace(S.saga_lstm_gather_workspace_size(g.plan, H), device())
    for a, b in zip(cuts[:-1], cuts[1:]):
        S.saga_lstm_gather_rows(g.plan, int(a), int(b), S.cmat(Pt), S.cmat(Wt), S.mat(out),
                                C.c_void_p(ws.data_ptr()), ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    assert np.array_equal(to_np(out), full)
    # a partial range leaves the other rows untouched
    out2 = dev_padded(np.full((n, H), 5.0))
    S.saga_lstm_gather_rows(g.plan, int(cuts[1]), int(cuts[3]), S.cmat(Pt), S.cmat(Wt), S.mat(out2),
                            C.c_void_p(ws.data_ptr()), ws.numel(), S.stream_handle())
    torch.cuda.synchronize()
    got = to_np(out2)
    inside = perm[cuts[1]:cuts[3]]
    outside = np.setdiff1d(np.arange(n), inside)
    assert np.array_equal(got[inside], full[inside])
    assert np.all(got[outside] == 5.0)
    with pytest.raises(S.SagaError):
        S.saga_lstm_gather_rows(g.plan, 3, 2, S.cmat(Pt), S.cmat(Wt), S.mat(out2),
                                C.c_void_p(ws.data_ptr()), ws.numel(), S.stream_handle())
