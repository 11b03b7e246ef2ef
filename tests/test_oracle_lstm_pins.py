"""Pins of the oracle's LSTM Gather (GraphSAGE row of Table I; Sec. 3.2,
Gather paragraph): an independent library LSTM (torch.nn.LSTM on the CPU in
float64, gate order i, f, g, o), closed forms, invariants, and planted
mistakes that each break a pin.  CPU only."""
import numpy as np
import pytest
import torch

from helpers import edges_to_csr, tiny_graphs
from oracle import saga_oracle as O


def _weights(F, H, seed):
    rng = np.random.default_rng(seed)
    a = 1.0 / np.sqrt(H)
    return (rng.uniform(-a, a, (F, 4 * H)), rng.uniform(-a, a, 4 * H),
            rng.uniform(-a, a, (H, 4 * H)), rng.uniform(-a, a, 4 * H))


def _torch_lstm_final(X_seq, W_ih, b_ih, W_hh, b_hh):
    H = W_hh.shape[0]
    m = torch.nn.LSTM(X_seq.shape[1], H).double()
    with torch.no_grad():
        m.weight_ih_l0.copy_(torch.from_numpy(np.ascontiguousarray(W_ih.T)))
        m.weight_hh_l0.copy_(torch.from_numpy(np.ascontiguousarray(W_hh.T)))
        m.bias_ih_l0.copy_(torch.from_numpy(b_ih))
        m.bias_hh_l0.copy_(torch.from_numpy(b_hh))
        _, (h, _) = m(torch.from_numpy(X_seq)[:, None, :])
    return h[0, 0].numpy()


def _graphs():
    out = [(name, n, *edges_to_csr(n, src, dst)[:2]) for name, n, src, dst in tiny_graphs()]
    from synth import configs as C

    g = C.build("sage_lstm", small=True)
    out.append(("rmat", g["num_vertices"], g["row_ptr"], g["col_idx"]))
    return out


@pytest.mark.parametrize("case", _graphs(), ids=lambda c: c[0])
def test_lstm_gather_equals_library_lstm(case):
    name, n, rp, col = case
    F, H = 6, 5
    X = np.random.default_rng(1).standard_normal((n, F))
    W_ih, b_ih, W_hh, b_hh = _weights(F, H, 2)
    d = np.diff(rp)
    rows = np.arange(n) if n <= 64 else np.unique(np.concatenate(
        [np.argsort(d)[-3:], np.flatnonzero(d == 0)[:2], np.arange(0, n, n // 20)]))
    got = O.lstm_gather(rp, col, X, W_ih, b_ih, W_hh, b_hh, rows=rows)
    for k, v in enumerate(rows):
        nb = col[rp[v]:rp[v + 1]]
        want = np.zeros(H) if len(nb) == 0 else _torch_lstm_final(X[nb], W_ih, b_ih, W_hh, b_hh)
        assert np.allclose(got[k], want, rtol=0, atol=1e-12), (name, v)


def test_lstm_one_neighbour_closed_form():
    # one step from h = c = 0: h = s(o) tanh(s(i) tanh(g)), z = x W_ih + b
    F, H = 4, 3
    W_ih, b_ih, W_hh, b_hh = _weights(F, H, 5)
    x = np.array([[0.5, -1.0, 2.0, 0.25], [1.0, 1.0, 1.0, 1.0]])
    rp, col = np.array([0, 1, 1]), np.array([1])
    got = O.lstm_gather(rp, col, x, W_ih, b_ih, W_hh, b_hh)
    z = x[1] @ W_ih + b_ih + b_hh
    s = lambda t: 1 / (1 + np.exp(-t))  # noqa: E731
    want = s(z[3 * H:]) * np.tanh(s(z[:H]) * np.tanh(z[2 * H:3 * H]))
    assert np.allclose(got[0], want, rtol=0, atol=1e-15)
    assert np.array_equal(got[1], np.zeros(H))     # empty row


def test_lstm_zero_weights_give_zero():
    # all gates pre-activate at 0: g = 0 keeps c = 0, so h = 0 whatever the input
    rp, col = np.array([0, 3]), np.array([0, 0, 0])
    X = np.ones((1, 4))
    z = np.zeros
    assert np.array_equal(O.lstm_gather(rp, col, X, z((4, 8)), z(8), z((2, 8)), z(8)), z((1, 2)))


def test_lstm_reads_the_sequence_in_csr_order():
    F, H = 3, 4
    W_ih, b_ih, W_hh, b_hh = _weights(F, H, 7)
    X = np.random.default_rng(8).standard_normal((4, F))
    a = O.lstm_gather(np.array([0, 3]), np.array([1, 2, 3]), X, W_ih, b_ih, W_hh, b_hh)
    b = O.lstm_gather(np.array([0, 3]), np.array([3, 2, 1]), X, W_ih, b_ih, W_hh, b_hh)
    assert not np.allclose(a, b)
    assert np.allclose(b[0], _torch_lstm_final(X[[3, 2, 1]], W_ih, b_ih, W_hh, b_hh), atol=1e-12)


def test_sage_lstm_layer_composition_and_equivariance():
    from synth import configs as C

    g = C.build("sage_lstm", small=True)
    rows = np.arange(0, g["num_vertices"], 37)
    y = O.sage_lstm_layer_of(g, rows=rows)
    A = O.lstm_gather(g["row_ptr"], g["col_idx"], g["X"], g["W_ih"], g["b_ih"], g["W_hh"],
                      g["b_hh"], rows=rows)
    want = np.concatenate([g["X"][rows].astype(np.float64), A], 1) @ g["W"].astype(np.float64) + g["b"]
    assert np.allclose(y, want, rtol=0, atol=1e-12)
    # relabel vertices (each row keeps its neighbour order): outputs permute
    n = g["num_vertices"]
    pi = np.random.default_rng(3).permutation(n)        # new id of old vertex v is pi[v]
    inv = np.argsort(pi)
    rp, col = g["row_ptr"], g["col_idx"]
    d = np.diff(rp)[inv]
    rp2 = np.concatenate([[0], np.cumsum(d)])
    col2 = np.concatenate([pi[col[rp[v]:rp[v + 1]]] for v in inv])
    g2 = dict(g, row_ptr=rp2, col_idx=col2, X=g["X"][inv])
    y2 = O.sage_lstm_layer_of(g2, rows=pi[rows])
    assert np.allclose(y2, y, rtol=0, atol=1e-12)


# planted mistakes in the LSTM step: each breaks the library-LSTM pin
def _swap_if(z, c):
    H = c.shape[0]
    z = np.concatenate([z[H:2 * H], z[:H], z[2 * H:]])
    return _cell(z, c)


def _no_forget(z, c):
    H = c.shape[0]
    return _cell(np.concatenate([z[:H], np.full(H, 50.0), z[2 * H:]]), c * 0)


def _no_output_gate(z, c):
    H = c.shape[0]
    return _cell(np.concatenate([z[:3 * H], np.full(H, 50.0)]), c)


_cell = O.lstm_cell
LSTM_MUTANTS = {"swap_i_f": _swap_if, "no_forget": _no_forget, "no_output_gate": _no_output_gate}


@pytest.mark.parametrize("mutant", sorted(LSTM_MUTANTS))
def test_planted_lstm_mistake_is_caught(mutant, monkeypatch):
    monkeypatch.setattr(O, "lstm_cell", LSTM_MUTANTS[mutant])
    with pytest.raises(AssertionError):
        test_lstm_gather_equals_library_lstm(_graphs()[-1])
