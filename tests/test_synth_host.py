"""The seeded synthetic inputs (the workloads' stand-ins for the paper's
datasets, Table II): the seed convention, determinism, the edge counts and
graph rules the input recipe states, on the CPU."""
import numpy as np
import pytest

from synth import configs as Cfg
from synth import graphs as G

WORKLOADS = ["gcn_er", "gat_ba", "sage_rmat", "gated_rgg", "gcn_rmat", "sage_lstm", "rgcn_rmat"]


def _edges(d):
    rp = d["row_ptr"].astype(np.int64)
    dst = np.repeat(np.arange(d["num_vertices"]), np.diff(rp))
    return d["col_idx"].astype(np.int64), dst


def test_seed_convention():
    ss = G.seed_seq(5, 4)
    assert ss.entropy == 200900804 and ss.spawn_key == (5, 4)
    a = G.rng_for(3, 1).standard_normal(4)
    b = np.random.Generator(np.random.PCG64(np.random.SeedSequence(200900804, spawn_key=(3, 1))))
    assert np.array_equal(a, b.standard_normal(4))


@pytest.mark.parametrize("name", WORKLOADS)
def test_small_variants_are_deterministic_canonical_csr(name):
    a, b = Cfg.build(name, small=True), Cfg.build(name, small=True)
    assert sorted(a) == sorted(b)
    for k in a:  # byte identity (padding columns hold NaN by design)
        if isinstance(a[k], np.ndarray):
            assert a[k].dtype == b[k].dtype and a[k].tobytes() == b[k].tobytes(), k
    rp, col = a["row_ptr"], a["col_idx"]
    assert rp[0] == 0 and rp[-1] == a["num_edges"] == len(col) and np.all(np.diff(rp) >= 0)
    assert col.min() >= 0 and col.max() < a["num_vertices"]
    # within a row, sources ascend (the canonical order of the in-CSR)
    starts = np.zeros(len(col), bool)
    starts[rp[:-1][np.diff(rp) > 0]] = True
    assert np.all((np.diff(col.astype(np.int64)) >= 0) | starts[1:])


def test_er_distinct_pairs_plus_one_self_loop_each():
    d = Cfg.build("gcn_er")
    assert d["num_vertices"] == 2000 and d["num_edges"] == 12000
    src, dst = _edges(d)
    loops = src == dst
    assert loops.sum() == 2000 and np.array_equal(np.sort(src[loops]), np.arange(2000))
    pairs = src[~loops] * 2000 + dst[~loops]
    assert len(np.unique(pairs)) == 10000


def test_ba_symmetric_with_self_loops():
    d = Cfg.build("gat_ba")
    assert d["num_vertices"] == 20000 and d["num_edges"] == 219950
    src, dst = _edges(d)
    loops = src == dst
    assert loops.sum() == 20000
    fwd = np.sort(src[~loops] * 20000 + dst[~loops])
    bwd = np.sort(dst[~loops] * 20000 + src[~loops])
    assert np.array_equal(fwd, bwd)  # every edge stored in both directions


def test_torus_rgg_symmetric_within_radius_degree_twelve():
    d = Cfg.build("gated_rgg")
    n = d["num_vertices"]
    src, dst = _edges(d)
    assert not np.any(src == dst)
    assert np.array_equal(np.sort(src * n + dst), np.sort(dst * n + src))
    assert abs(d["num_edges"] / n - 12.0) < 0.3
    assert d["E_feat"].shape[0] == d["num_edges"]


@pytest.mark.parametrize("name,scale,avg", [("sage_rmat", 17, 16), ("rgcn_rmat", 18, 16)])
def test_rmat_edge_count_and_relabelled(name, scale, avg):
    d = Cfg.build(name)
    n = 1 << scale
    assert d["num_vertices"] == n and d["num_edges"] == avg * n
    # the relabelling leaves no trace of R-MAT's low-id hubs: the busiest
    # sources are spread over the id range
    src, _ = _edges(d)
    top = np.argsort(-np.bincount(src, minlength=n), kind="stable")[:64]
    assert np.median(top) > n / 8


def test_gcn_rmat_recipe_at_reduced_scale():
    """The 2^21 workload's recipe (50 edges per vertex, relabelled, one
    self-loop per vertex) at scale 13."""
    d = Cfg.build("gcn_rmat", small=True)
    n = d["num_vertices"]
    assert n == 1 << 13 and d["num_edges"] == 51 * n
    src, dst = _edges(d)
    assert np.sum(src == dst) >= n  # the added loops, plus any R-MAT draws
