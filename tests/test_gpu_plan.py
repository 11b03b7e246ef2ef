"""Graph layout built on the GPU equals the oracle's, bit for bit."""
import numpy as np
import pytest

from gpu_util import graph, lib
from helpers import edges_to_csr, tiny_graphs
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
