"""The 2^21-vertex R-MAT GCN (50 edges per vertex + self-loops, 602 -> 128
-> 41) at full size, in the launch configuration the benchmark times.

The oracle cannot evaluate 2M rows, so it checks: the whole plan bit for bit
(integer layout), sampled output rows of layer 1 (including the largest hub
and split rows), sampled rows of the two-layer model whose two-hop
neighbourhoods are small, layer 2 on its hub and split rows fed the GPU's
own layer-1 output, and properties that hold at any size (finite outputs,
run-to-run identical bytes).  The benchmark's step is checked both stage by
stage and with the plan's row order on a second stream (the configuration
its headline number is timed in)."""
import numpy as np
import pytest
import torch

from gpu_util import dev_int, lib, to_np
from helpers import BF16_TOL, FP32_TOL, rel_err, rel_err_terms
from oracle import saga_oracle as O
from synth import configs as C
from synth import tensors as T

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(scope="module")
def big():
    print("generating the 2^21-vertex R-MAT workload ...", flush=True)
    g = C.build("gcn_rmat")
    print(f"V={g['num_vertices']} E={g['num_edges']}", flush=True)
    return g


@pytest.fixture(scope="module")
def dev_graph(big):
    S = lib()
    rp = dev_int(big["row_ptr"])
    col = dev_int(big["col_idx"])
    return S.Graph(rp, col)


def _samples(g, k=48, seed=0):
    rp = g["row_ptr"].astype(np.int64)
    d = np.diff(rp)
    rng = np.random.default_rng(seed)
    rows = set(rng.integers(0, len(d), k).tolist())
    rows.add(int(np.argmax(d)))                    # the largest hub
    split = np.flatnonzero(d > 512)
    rows.update(rng.choice(split, 8, replace=False).tolist())
    rows.update(np.flatnonzero(d == d.min())[:4].tolist())
    return np.array(sorted(rows))


def _small_two_hop(g, k=24, limit=40000, seed=1):
    rp = g["row_ptr"].astype(np.int64)
    col = g["col_idx"]
    d = np.diff(rp)
    rng = np.random.default_rng(seed)
    out = []
    for v in rng.permutation(len(d)):
        nb = col[rp[v]:rp[v + 1]]
        if d[nb].sum() <= limit:
            out.append(int(v))
        if len(out) == k:
            break
    return np.array(sorted(out))


def _layer_mag(rp, col, X, W, b, rows):
    """Magnitude of the terms summed into each pre-activation output of a
    GCN layer: the layer on |X|, |W|, |b| without the activation."""
    return O.gcn_layer(rp, col, np.abs(X), np.abs(W), np.abs(b), "none", rows=rows)


def _model_mag(g, X, W1, W2, rows):
    """Magnitude of the terms of the two-layer model's outputs: the model on
    |X|, |W1|, |W2|, |b1|, |b2| (its ReLU is the identity there)."""
    return O.gcn_2layer(dict(g, b1=np.abs(g["b1"]), b2=np.abs(g["b2"])), X=np.abs(X),
                        W1=np.abs(W1), W2=np.abs(W2), rows=rows)


def _hub_rows(g, k_top=4, k_split=4, seed=5):
    """The largest in-degree rows and a few other split rows."""
    d = np.diff(g["row_ptr"].astype(np.int64))
    top = np.argsort(-d, kind="stable")[:k_top]
    split = np.setdiff1d(np.flatnonzero(d > 512), top)
    rng = np.random.default_rng(seed)
    return np.sort(np.concatenate([top, rng.choice(split, k_split, replace=False)]))


def test_full_plan_bit_exact(big, dev_graph):
    got = {k: v.cpu().numpy().astype(np.int64) for k, v in dev_graph.arrays().items()}
    p = dev_graph.plan
    print("oracle plan ...", flush=True)
    want = O.plan(big["row_ptr"], big["col_idx"], big["num_vertices"], p.seg_len, p.block_cost,
                  p.row_cost)
    for k in ("d_in", "d_out", "perm", "row_seg_first", "seg_row", "seg_beg", "seg_end",
              "block_ptr"):
        assert np.array_equal(got[k], want[k]), k
    assert dev_graph.counts.n_split == want["n_split"]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_full_gcn_sampled(big, dev_graph, dtype):
    from paper_2009_00804_amd import layers as LY

    g = big
    f_in, hid, f_out = g["dims"]
    if dtype == "f32":
        X = torch.from_numpy(g["X"]).cuda()[:, :f_in]   # ld 604: 16-byte rows
        Xo = g["X"][:, :f_in]
        W1, W2 = g["W1"], g["W2"]
        tdt, tol = torch.float32, FP32_TOL
    else:
        C.add_bf16_variant(g)
        bits = torch.from_numpy(g["X_bf16"].view(np.int16)).view(torch.bfloat16)
        X = bits.cuda()[:, :f_in]                        # ld 608
        Xo = T.bf16_to_f32(g["X_bf16"][:, :f_in])
        W1, W2 = g["W1_bf"], g["W2_bf"]
        tdt, tol = torch.bfloat16, BF16_TOL
    model = LY.gcn2(dev_graph, torch.from_numpy(W1), torch.from_numpy(g["b1"]),
                    torch.from_numpy(W2), torch.from_numpy(g["b2"]), dtype=tdt, out_ld=44 if dtype == "f32" else 48)
    print(f"running the {dtype} forward on the GPU", flush=True)
    y = LY.run(model, X).clone()
    h1 = model[0].out
    torch.cuda.synchronize()
    assert torch.isfinite(y.float()).all()
    y_again = LY.run(model, X)
    torch.cuda.synchronize()
    assert torch.equal(y, y_again)                 # deterministic bytes

    rp, col = g["row_ptr"], g["col_idx"]
    rows = _samples(g)
    print(f"oracle layer 1 on {len(rows)} sampled rows", flush=True)
    ref1 = O.gcn_layer(rp, col, Xo, W1, g["b1"], "relu", rows=rows)
    mag1 = _layer_mag(rp, col, Xo, W1, g["b1"], rows)
    got1 = to_np(h1[torch.from_numpy(rows).cuda()])
    e1 = rel_err(got1, ref1)
    e1t = rel_err_terms(got1, ref1, mag1)
    rows2 = _small_two_hop(g)
    print(f"oracle two layers on {len(rows2)} sampled rows", flush=True)
    ref2 = O.gcn_2layer(dict(g, X=Xo), X=Xo, W1=W1, W2=W2, rows=rows2)
    got2 = to_np(y[torch.from_numpy(rows2).cuda()])
    e2 = rel_err(got2, ref2)
    e2t = rel_err_terms(got2, ref2, _model_mag(g, Xo, W1, W2, rows2))
    print(f"{dtype}: layer-1 sampled err {e1:.3e} (per-element terms {e1t:.3e}), two-layer "
          f"sampled err {e2:.3e} (terms {e2t:.3e})", flush=True)
    assert e1 <= tol
    assert e1t <= tol
    assert e2 <= tol
    assert e2t <= tol


@pytest.mark.parametrize("split", [False, True], ids=["stage_by_stage", "pipelined"])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_full_bench_step_sampled(big, dtype, split):
    """The op-level call sequence the benchmark times (plan, GEMM, fused
    gather, GEMM, fused gather, with its buffers and leading dimensions) and
    the unfused layer-1 aggregation it is compared with, on sampled rows;
    stage by stage and with the plan's row order on a second stream
    overlapping the first transform (the configuration the headline number
    is timed in)."""
    import bench

    g = big
    if dtype == "bf16":
        C.add_bf16_variant(g)
        Xo = T.bf16_to_f32(g["X_bf16"][:, :g["dims"][0]])
        W1, W2, tol = g["W1_bf"], g["W2_bf"], BF16_TOL
    else:
        Xo = g["X"][:, :g["dims"][0]]
        W1, W2, tol = g["W1"], g["W2"], FP32_TOL
    step = bench.Step(g, dtype, torch.device("cuda:0"))
    step.split = split
    print(f"bench step ({dtype}, split={split}) on the GPU", flush=True)
    step.run()
    torch.cuda.synchronize()
    y = step.Y.clone()
    step.run()
    torch.cuda.synchronize()
    assert torch.equal(y, step.Y)                  # deterministic bytes
    assert torch.isfinite(y.float()).all()
    rp, col = g["row_ptr"], g["col_idx"]
    rows = _samples(g, seed=3)
    rsel = torch.from_numpy(rows).cuda()
    print(f"oracle layer 1 on {len(rows)} sampled rows", flush=True)
    ref1 = O.gcn_layer(rp, col, Xo, W1, g["b1"], "relu", rows=rows)
    got1 = to_np(step.H1[rsel])
    e1 = rel_err(got1, ref1)
    e1t = rel_err_terms(got1, ref1, _layer_mag(rp, col, Xo, W1, g["b1"], rows))
    # layer 2 on its hub and split rows (up to hundreds of thousands of
    # in-edges), fed the layer-1 output the GPU produced
    hubs = _hub_rows(g)
    print(f"oracle layer 2 on {len(hubs)} hub / split rows from the GPU's H1", flush=True)
    H1 = to_np(step.H1)
    ref_h = O.gcn_layer(rp, col, H1, W2, g["b2"], "none", rows=hubs)
    got_h = to_np(y[torch.from_numpy(hubs).cuda()])
    eh = rel_err(got_h, ref_h)
    eht = rel_err_terms(got_h, ref_h, _layer_mag(rp, col, H1, W2, g["b2"], hubs))
    del H1
    print("unfused layer-1 aggregation on the GPU", flush=True)
    step.setup_unfused()
    hu = step.run_unfused1()
    torch.cuda.synchronize()
    eu = rel_err(to_np(hu[rsel]), ref1)
    step.free_unfused()
    rows2 = _small_two_hop(g, seed=4)
    print(f"oracle two layers on {len(rows2)} sampled rows", flush=True)
    ref2 = O.gcn_2layer(dict(g, X=Xo), X=Xo, W1=W1, W2=W2, rows=rows2)
    got2 = to_np(y[torch.from_numpy(rows2).cuda()])
    e2 = rel_err(got2, ref2)
    e2t = rel_err_terms(got2, ref2, _model_mag(g, Xo, W1, W2, rows2))
    print(f"{dtype} split={split}: layer-1 err {e1:.3e} (per-element terms {e1t:.3e}), "
          f"unfused layer-1 err {eu:.3e}, layer-2 hub rows err {eh:.3e} (terms {eht:.3e}), "
          f"two-layer err {e2:.3e} (terms {e2t:.3e})", flush=True)
    assert e1 <= tol
    assert e1t <= tol
    assert eu <= tol
    assert eh <= tol
    assert eht <= tol
    assert e2 <= tol
    assert e2t <= tol
    del step
    torch.cuda.empty_cache()


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_full_bench_step_fused_sampled(big, dtype):
    """The benchmark's step with layer 2's transform fused into layer 1's
    Gather (and the plan's row order on a second stream): layer 2's
    transformed rows Z2 = d_out^-1/2 (H1 W2) on sampled rows (hubs and split
    rows, whose transform runs in the combine, included) against the
    oracle's layer 1 and product, and the two-layer output on rows with small
    two-hop neighbourhoods."""
    import bench

    g = big
    if dtype == "bf16":
        C.add_bf16_variant(g)
        Xo = T.bf16_to_f32(g["X_bf16"][:, :g["dims"][0]])
        W1, W2, tol = g["W1_bf"], g["W2_bf"], BF16_TOL
    else:
        Xo = g["X"][:, :g["dims"][0]]
        W1, W2, tol = g["W1"], g["W2"], FP32_TOL
    step = bench.Step(g, dtype, torch.device("cuda:0"))
    step.split = True
    step.fused = True
    print(f"bench step ({dtype}, pipelined, fused) on the GPU", flush=True)
    step.run()
    torch.cuda.synchronize()
    y = step.Y.clone()
    z2 = torch.cat([step.Z2, step.Z2t], dim=1) if step.split2 else step.Z2
    z2 = z2.clone()
    step.run()
    torch.cuda.synchronize()
    assert torch.equal(y, step.Y)                  # deterministic bytes
    rp, col = g["row_ptr"], g["col_idx"]
    rows = _samples(g, seed=6)
    print(f"oracle layer 1 and the layer-2 product on {len(rows)} sampled rows", flush=True)
    h1 = O.gcn_layer(rp, col, Xo, W1, g["b1"], "relu", rows=rows)
    s_out = O.degree_scale(O.out_degrees(col, g["num_vertices"]))[rows]
    ref_z = O.dense(h1, W2) * s_out[:, None]
    mag_z = O.dense(np.abs(_layer_mag(rp, col, Xo, W1, g["b1"], rows)), np.abs(W2)) * s_out[:, None]
    got_z = to_np(z2[torch.from_numpy(rows).cuda()])
    ez, ezt = rel_err(got_z, ref_z), rel_err_terms(got_z, ref_z, mag_z)
    rows2 = _small_two_hop(g, seed=7)
    print(f"oracle two layers on {len(rows2)} sampled rows", flush=True)
    ref2 = O.gcn_2layer(dict(g, X=Xo), X=Xo, W1=W1, W2=W2, rows=rows2)
    got2 = to_np(y[torch.from_numpy(rows2).cuda()])
    e2 = rel_err(got2, ref2)
    e2t = rel_err_terms(got2, ref2, _model_mag(g, Xo, W1, W2, rows2))
    print(f"{dtype} fused: Z2 err {ez:.3e} (terms {ezt:.3e}), two-layer err {e2:.3e} "
          f"(terms {e2t:.3e})", flush=True)
    assert ez <= tol and ezt <= tol
    assert e2 <= tol and e2t <= tol
    del step
    torch.cuda.empty_cache()
