"""Benchmark: one step = one full pass of the SAGA-NN hot path of a 2-layer
GCN on the 2^21-vertex R-MAT graph (50 edges per vertex + self-loops,
106,954,752 stored edges, features 602 -> 128 -> 41):

    graph layout (plan: degrees, degree order, segments, row blocks)
    layer 1: ApplyVertex-pre  Z1 = d_out^-1/2 (X W1)          (MFMA GEMM)
             Scatter+ApplyEdge+Gather+ApplyVertex-post
                              H1 = ReLU(d_in^-1/2 sum Z1_u + b1)
    layer 2: Z2 = d_out^-1/2 (H1 W2);  Y = d_in^-1/2 sum Z2_u + b2

Inputs are resident in HBM before the timed region.  ``value`` is layer
throughput in edges/s: (stored edges x 2 layers) / step time.  Prints one
JSON line (rank 0, one GPU).
"""
from __future__ import annotations

import argparse
import ctypes as C
import hashlib
import json
import os
import statistics
import sys
import time
import types

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM = 8.0e12          # bytes/s
PEAK_MFMA = {"f32": 157.3e12, "bf16": 2516.6e12}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def src_sha(name):
    p = os.path.join(ROOT, "paper_2009_00804_amd", "csrc", name)
    with open(p, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def load_traffic(kernel, dtype):
    """Per-launch HBM bytes of `kernel` from the counter summary in
    profiles/, if it was taken on the current kernel source."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(p):
        return None
    try:
        with open(p) as f:
            rec = json.load(f)
        e = rec.get(f"{kernel}:{dtype}")
        if not e or e.get("src_sha") != src_sha(e["source"]):
            return None
        return e["bytes_per_launch"]
    except Exception:
        return None


class Step:
    """Preallocated buffers and the op-level call sequence of one step."""

    def __init__(self, g, dtype, dev):
        import torch

        import paper_2009_00804_amd.saga as S

        self.S = S
        self.torch = torch
        self.dtype = dtype
        tdt = torch.float32 if dtype == "f32" else torch.bfloat16
        self.tdt = tdt
        f_in, hid, f_out = g["dims"]
        self.dims = g["dims"]
        self.V = g["num_vertices"]
        self.E = g["num_edges"]
        self.rp = torch.from_numpy(g["row_ptr"]).to(dev)
        self.col = torch.from_numpy(g["col_idx"]).to(dev)
        if dtype == "f32":
            self.X = torch.from_numpy(g["X"]).to(dev)[:, :f_in]
            W1, W2 = g["W1"], g["W2"]
        else:
            self.X = torch.from_numpy(g["X_bf16"].view("int16")).view(torch.bfloat16).to(dev)[:, :f_in]
            W1, W2 = g["W1_bf"], g["W2_bf"]
        self.W1 = torch.from_numpy(W1).to(dev).to(tdt)
        self.W2 = torch.from_numpy(W2).to(dev).to(tdt)
        self.b1 = torch.from_numpy(g["b1"]).to(dev)
        self.b2 = torch.from_numpy(g["b2"]).to(dev)
        es = 4 if dtype == "f32" else 2
        al = 16 // es
        ld = lambda c: (c + al - 1) // al * al  # noqa: E731
        self.Z1 = torch.empty((self.V, S.gather_ld(hid, es)), dtype=tdt, device=dev)[:, :hid]
        self.H1_base = torch.empty((self.V, ld(hid)), dtype=tdt, device=dev)
        self.H1 = self.H1_base[:, :hid]
        # Z2 rows longer than one 128-byte line but not whole lines (41 float32
        # columns) are written as two matrices: the whole-line columns and
        # the rest, each gathered by its own call (what saga_layer does)
        per_line = 128 // es
        self.split2 = f_out // per_line * per_line if f_out > per_line and f_out % per_line else 0
        if self.split2:
            self.Z2 = torch.empty((self.V, S.gather_ld(self.split2, es)), dtype=tdt,
                                  device=dev)[:, :self.split2]
            rest = f_out - self.split2
            self.Z2t = torch.empty((self.V, S.gather_ld(rest, es)), dtype=tdt, device=dev)[:, :rest]
        else:
            self.Z2 = torch.empty((self.V, S.gather_ld(f_out, es)), dtype=tdt, device=dev)[:, :f_out]
        self.Y = torch.empty((self.V, ld(f_out)), dtype=tdt, device=dev)[:, :f_out]
        self.graph = S.Graph(self.rp, self.col)     # allocates + builds + checks once
        self.plan_ws = self.graph.ws
        p = self.graph.plan
        op = S.saga_edge_op()
        self.op1 = S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_SUM, S.dtype_code(tdt), 1, 0, 1, 0.0,
                                  S.SAGA_ACT_RELU)
        self.op2 = S.saga_edge_op(S.SAGA_MSG_COPY, S.SAGA_RED_SUM, S.dtype_code(tdt), 1, 0, 1, 0.0,
                                  S.SAGA_ACT_NONE)
        del op
        n1 = S.saga_gather_workspace_size(p, self.op1, hid)
        n2 = S.saga_gather_workspace_size(p, self.op2, f_out)
        self.gws = S.workspace(max(n1, n2), dev)
        self.gop = S.saga_gemm_op(S.dtype_code(tdt), S.SAGA_GEMM_PLAIN, S.SAGA_ACT_NONE, p.d_out)
        self.gop2 = S.saga_gemm_op(S.dtype_code(tdt), S.SAGA_GEMM_PLAIN, S.SAGA_ACT_NONE, p.d_out)
        if self.split2:
            self.gop2.split_col = self.split2
            self.gop2.tail = S.mat(self.Z2t)
        m1 = S.saga_apply_vertex_workspace_size(self.gop, self.W1.shape[0], 0, self.W1.shape[1])
        m2 = S.saga_apply_vertex_workspace_size(self.gop, self.W2.shape[0], 0, self.W2.shape[1])
        self.mws = S.workspace(max(m1, m2), dev)
        self.none = S.saga_cmat(None, 0, 0, 0)
        self.in1 = S.saga_edge_inputs()
        self.in1.src = S.cmat(self.Z1)
        self.in1.bias = self.b1.data_ptr()
        self.in2 = S.saga_edge_inputs()
        self.in2.src = S.cmat(self.Z2)
        self.in2.bias = self.b2.data_ptr()
        self.out2 = S.mat(self.Y)
        if self.split2:
            sp = self.split2
            self.out2 = S.mat(self.Y[:, :sp])
            self.in2t = S.saga_edge_inputs()
            self.in2t.src = S.cmat(self.Z2t)
            self.in2t.bias = self.b2[sp:].data_ptr()
            self.out2t = S.mat(self.Y[:, sp:])
        self.stream = torch.cuda.current_stream()
        self.sh = S.stream_handle(self.stream)
        self.names = ["plan", "gemm1", "gather1", "gemm2", "gather2"]
        # cross-stage fusion: layer 1's Gather with layer 2's transform done
        # in its last slice pass writes Z2 (H1 lives only in the call's
        # workspace; no separate gemm2)
        self.fused = False
        self.nx = S.saga_next_transform()
        self.nx.w = S.cmat(self.W2)
        self.nx.row_scale_deg = p.d_out
        if self.split2:
            self.nx.split_col = self.split2
            self.nx.tail = S.mat(self.Z2t)
        self.xws = S.workspace(S.saga_gather_transform_workspace_size(p, self.op1, hid), dev)
        self.ev = None
        self.uws = None
        # stage pipelining: the plan's row-order branch on a second stream
        # (default priority) while the d_out-scaled transform runs here
        self.split = False
        self.join_early = False
        self.side = torch.cuda.Stream()
        self.side_sh = S.stream_handle(self.side)
        self.fork, self.join = torch.cuda.Event(), torch.cuda.Event()
        self.fork.record(self.stream)
        self.join.record(self.stream)  # creates both events

    def setup_unfused(self):
        """Workspace (the E x F edge tensor) and output of the unfused layer-1
        aggregation; allocated only when the fused/unfused comparison runs."""
        S, torch = self.S, self.torch
        hid = self.dims[1]
        n = S.saga_unfused_workspace_size(self.graph.plan, self.op1, hid)
        self.uws = S.workspace(n, self.H1.device)
        self.Hu = torch.empty_like(self.H1_base)[:, :hid]

    def run_unfused1(self):
        """Layer-1 Scatter+ApplyEdge+Gather, unfused (Fig. 7a): index-select
        into the edge tensor, then the segment reduction, on the same Z1."""
        S = self.S
        S.saga_scatter_gather_unfused(self.graph.plan, self.op1, self.in1, S.mat(self.Hu),
                                      C.c_void_p(self.uws.data_ptr()), self.uws.numel(), self.sh)
        return self.Hu

    def free_unfused(self):
        self.uws = None
        self.Hu = None

    def run(self, events=None):
        S = self.S
        g = self.graph
        ev = events
        if ev:
            ev[0].record(self.stream)
        if self.split:
            # out-degrees here, row order on the side stream; the transform
            # below waits for d_out only and overlaps the row order
            S.saga_plan_build_split(g.num_dst, g.num_src, g.num_edges, C.c_void_p(self.rp.data_ptr()),
                                    C.c_void_p(self.col.data_ptr()), g.opts,
                                    C.c_void_p(self.plan_ws.data_ptr()), self.plan_ws.numel(),
                                    self.sh, self.side_sh, C.c_void_p(self.fork.cuda_event),
                                    C.c_void_p(self.join.cuda_event))
        else:
            S.saga_plan_build(g.num_dst, g.num_src, g.num_edges, C.c_void_p(self.rp.data_ptr()),
                              C.c_void_p(self.col.data_ptr()), g.opts,
                              C.c_void_p(self.plan_ws.data_ptr()), self.plan_ws.numel(), self.sh)
        if ev:
            ev[1].record(self.stream)
        p = g.plan
        if self.split and self.join_early:
            # both plan branches finish before the transform, which then has
            # the CUs to itself
            self.stream.wait_event(self.join)
        S.saga_apply_vertex(self.gop, S.cmat(self.X), S.cmat(self.W1), self.none, self.none, None,
                            None, S.mat(self.Z1), C.c_void_p(self.mws.data_ptr()), self.mws.numel(),
                            self.sh)
        if self.split and not self.join_early:
            self.stream.wait_event(self.join)
        if ev:
            ev[2].record(self.stream)
        if self.fused:
            S.saga_scatter_apply_edge_gather_transform(p, self.op1, self.in1, self.nx, S.mat(self.Z2),
                                                       C.c_void_p(self.xws.data_ptr()), self.xws.numel(),
                                                       self.sh)
            if ev:
                ev[3].record(self.stream)
                ev[4].record(self.stream)
        else:
            S.saga_scatter_apply_edge_gather(p, self.op1, self.in1, S.mat(self.H1),
                                             C.c_void_p(self.gws.data_ptr()), self.gws.numel(), self.sh)
            if ev:
                ev[3].record(self.stream)
            S.saga_apply_vertex(self.gop2, S.cmat(self.H1), S.cmat(self.W2), self.none, self.none,
                                None, None, S.mat(self.Z2), C.c_void_p(self.mws.data_ptr()),
                                self.mws.numel(), self.sh)
            if ev:
                ev[4].record(self.stream)
        S.saga_scatter_apply_edge_gather(p, self.op2, self.in2, self.out2,
                                         C.c_void_p(self.gws.data_ptr()), self.gws.numel(), self.sh)
        if self.split2:
            S.saga_scatter_apply_edge_gather(p, self.op2, self.in2t, self.out2t,
                                             C.c_void_p(self.gws.data_ptr()), self.gws.numel(),
                                             self.sh)
        if ev:
            ev[5].record(self.stream)


def algorithmic(step, stage):
    """Algorithmic work of one launch of a stage: (bytes, flops).

    Gather: compulsory bytes -- every CSR index once (4 B/edge), row_ptr,
    the source matrix once and the output once (each unique byte once).
    GEMM: flops 2 M K N; bytes = A + W + output once."""
    V, E = step.V, step.E
    f_in, hid, f_out = step.dims
    es = 4 if step.dtype == "f32" else 2
    if stage == "gather1":
        return E * 4 + (V + 1) * 4 + 2 * V * hid * es, 2 * E * hid
    if stage == "gather2":
        return E * 4 + (V + 1) * 4 + 2 * V * f_out * es, 2 * E * f_out
    if stage == "gemm1":
        return V * f_in * es + f_in * hid * es + V * hid * es, 2 * V * f_in * hid
    if stage == "gemm2":
        return V * hid * es + hid * f_out * es + V * f_out * es, 2 * V * hid * f_out
    return (V + 1) * 4 + E * 4 + 3 * V * 4, 0


def noreuse_bytes(step, stage):
    """Bytes the gather moves through the memory hierarchy if no source row
    were reused from cache: per edge the index and the full source row."""
    V, E = step.V, step.E
    f_in, hid, f_out = step.dims
    es = 4 if step.dtype == "f32" else 2
    F = hid if stage == "gather1" else f_out
    row = (F * es + 15) // 16 * 16
    return E * (4 + row) + (V + 1) * 4 + V * F * es


def stage_rooflines(V, E, dims, dtype, mean):
    """Every stage of the step against its roofline: the GEMMs against the
    dtype's dense MFMA peak (and HBM for their compulsory bytes), the
    Gathers against 8 TB/s for their compulsory bytes, and, where the
    counter record in profiles/ matches the kernel source, for the measured
    FETCH_SIZE + WRITE_SIZE traffic."""
    shim = types.SimpleNamespace(V=V, E=E, dims=dims, dtype=dtype)
    out = {}
    for n in ("gemm1", "gather1", "gemm2", "gather2"):
        t = mean[n] * 1e-3
        byts, flops = algorithmic(shim, n)
        d = {"ms": round(mean[n], 4), "compulsory_GBps": byts / t / 1e9,
             "compulsory_frac_of_8TBps": byts / t / PEAK_HBM}
        if n.startswith("gemm"):
            d["TFLOPs"] = flops / t / 1e12
            d["mfma_frac"] = flops / t / PEAK_MFMA[dtype]
        else:
            d["noreuse_GBps"] = noreuse_bytes(shim, n) / t / 1e9
        tr = load_traffic(n, dtype)
        if tr:
            d["counter_GBps"] = tr / t / 1e9
            d["counter_frac_of_8TBps"] = tr / t / PEAK_HBM
        out[n] = d
    return out


def time_step(step, steps, warmup):
    torch = step.torch
    for _ in range(warmup):
        step.run()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for k in range(steps):
        step.run(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = {n: [] for n in step.names}
    tot = []
    for e in evs:
        for i, n in enumerate(step.names):
            per[n].append(e[i].elapsed_time(e[i + 1]))
        tot.append(e[0].elapsed_time(e[5]))
    return wall, per, tot


def time_unfused(step, reps=3):
    """Mean time of the unfused layer-1 aggregation next to the fused one."""
    torch = step.torch
    step.setup_unfused()
    step.run_unfused1()
    torch.cuda.synchronize()
    e0 = torch.cuda.Event(enable_timing=True)
    e1 = torch.cuda.Event(enable_timing=True)
    e0.record(step.stream)
    for _ in range(reps):
        step.run_unfused1()
    e1.record(step.stream)
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / reps
    step.free_unfused()
    torch.cuda.empty_cache()
    return ms


SUITE = [  # the other workloads, one model each (Table I models at their configured sizes)
    ("gcn_er", "2-layer GCN, directed ER G(2000, 10000) + self-loops, 128->16->8"),
    ("gat_ba", "2-layer GAT, BA(20000, m=5) symmetrised + self-loops, 512->8x8->8x8 (mean)"),
    ("sage_rmat", "GraphSAGE-pool, R-MAT scale 17, 16 edges/vertex, 256->256"),
    ("gated_rgg", "gated edge MPNN + GRU, torus RGG(100000, expected degree 12), 64 (+16 edge)"),
    ("sage_lstm", "GraphSAGE-LSTM, R-MAT scale 17, 16 edges/vertex, 256 -> LSTM 128 -> 256"),
    ("rgcn_rmat", "R-GCN, R-MAT scale 18, 16 edges/vertex, 32 relation types (P(r) ~ 1/(r+1)), "
                  "128 -> 64, ReLU"),
]


def _padded(a, torch, dev):
    """Device copy of a float32 matrix with 16-byte-aligned rows."""
    a = torch.from_numpy(a)
    n, f = a.shape
    ld = (f + 3) // 4 * 4
    t = torch.zeros((n, ld), dtype=torch.float32, device=dev)
    t[:, :f] = a.to(dev)
    return t[:, :f]


def _oracle_model(name, g, rows=None):
    from oracle import saga_oracle as O

    if name == "gcn_er":
        return O.gcn_2layer(g, X=g["X"][:, :g["dims"][0]])
    if name == "gat_ba":
        return O.gat_2layer(g)
    if name == "sage_rmat":
        return O.sage_layer_of(g)
    if name == "sage_lstm":
        return O.sage_lstm_layer_of(g, rows=rows)
    if name == "rgcn_rmat":
        return O.rgcn_layer_of(g, rows=rows)
    return O.gated_layer_of(g)


# layers of each suite workload's model (the others have one)
SUITE_LAYERS = {"gcn_er": 2, "gat_ba": 2}
_SUITE_G = {}


def _suite_rows(name, g):
    """The bounded destination-row sample the oracle runs on for the
    workloads whose oracle loops over rows (and, for the LSTM, steps);
    None: the whole model."""
    import numpy as np

    if name not in ("sage_lstm", "rgcn_rmat"):
        return None
    return np.random.default_rng(7).choice(g["num_vertices"], 1500 if name == "sage_lstm" else 4000,
                                           replace=False)


def _suite_oracle_runs(args):
    """(runs, seconds): the oracle of one workload on one thread, repeated
    until `budget_s` has passed (at least once)."""
    name, budget_s = args
    from threadpoolctl import threadpool_limits

    g = _SUITE_G[name]
    rows = _suite_rows(name, g)
    runs, t = 0, 0.0
    with threadpool_limits(1):
        while runs == 0 or t < budget_s:
            t0 = time.perf_counter()
            _oracle_model(name, g, rows=rows)
            t += time.perf_counter() - t0
            runs += 1
    return runs, t


def suite_oracles(reps=3, budget_s=1.0):
    """The oracle of each suite workload, run before the GPU is touched
    (the all-cores leg forks worker processes): on one thread, the median
    of `reps` runs; and on every core of the affinity mask (at most 16),
    each worker process one thread repeating the whole evaluation for
    `budget_s`, the throughput summed over the workers."""
    import multiprocessing as mp

    import numpy as np

    from synth import configs as Cfg

    out = {}
    cores = max(1, min(len(os.sched_getaffinity(0)), 16))
    for name, _ in SUITE:
        g = Cfg.build(name)
        _SUITE_G.clear()
        _SUITE_G[name] = g
        rows = _suite_rows(name, g)
        work = SUITE_LAYERS.get(name, 1) * (g["num_edges"] if rows is None
                                             else int(np.diff(g["row_ptr"])[rows].sum()))
        sample = ("whole model, float64" if rows is None else
                  f"layer on {len(rows)} random destination rows ({work} in-edges), float64")
        t1 = statistics.median(_suite_oracle_runs((name, 0.0))[1] for _ in range(reps))
        rec = {"ms": t1 * 1e3, "edges_per_s": work / t1, "cores": 1, "kind": "oracle",
               "sample": f"{sample}, median of {reps} runs", "cpu_model": _cpu_model()}
        if cores > 1:
            with mp.get_context("fork").Pool(cores) as pool:
                res = pool.map(_suite_oracle_runs, [(name, budget_s)] * cores)
            rec["all_cores"] = {
                "edges_per_s": sum(r[0] * work / r[1] for r in res), "cores": cores,
                "sample": f"{cores} worker processes of one thread, each repeating the "
                          f"evaluation for {budget_s:g} s ({sum(r[0] for r in res)} runs)"}
        out[name] = rec
        log(f"suite oracle {name}: {t1 * 1e3:.1f} ms on one thread"
            + (f", {rec['all_cores']['edges_per_s']:.3e} edges/s on {cores} cores"
               if cores > 1 else ""))
    _SUITE_G.clear()
    return out


def _gemm_work(M, K, N, es=4):
    """(compulsory bytes, flops) of an M x K by K x N product: A, W and the
    output once; 2 M K N."""
    return (M * K + K * N + M * N) * es, 2 * M * K * N


def _gather_work(V, E, F_src, F_out, src_rows=None, per_edge_bytes=0, per_row_bytes=0,
                 flops_per_edge=None):
    """(compulsory bytes, flops) of a Gather: 4 B per CSR index, row_ptr, each
    source row once, the output once, plus the kernel's other inputs."""
    src_rows = V if src_rows is None else src_rows
    byts = (E * 4 + (V + 1) * 4 + src_rows * F_src * 4 + V * F_out * 4 + E * per_edge_bytes
            + V * per_row_bytes)
    return byts, E * (F_src if flops_per_edge is None else flops_per_edge)


def suite_stages(name, g, rel_counts=None):
    """The stages saga_layer runs for each layer of a workload (the order
    saga_trace_stages reports them in), with the algorithmic work of each:
    [[(stage, kind, bytes, flops), ...] per layer]; kind "mfma" for the
    dense transforms (priced against the float32 MFMA peak), "hbm" for the
    Gathers."""
    V, E = g["num_vertices"], g["num_edges"]
    G = lambda st, w: (st, "mfma", *w)  # noqa: E731
    A = lambda st, w: (st, "hbm", *w)   # noqa: E731
    if name == "gcn_er":
        f_in, hid, f_out = g["dims"]
        return [[G("transform", _gemm_work(V, f_in, hid)), A("gather", _gather_work(V, E, hid, hid))],
                [G("transform", _gemm_work(V, hid, f_out)), A("gather", _gather_work(V, E, f_out, f_out))]]
    if name == "gat_ba":
        K = g["heads"]
        f_in, F1 = g["W1"].shape
        F2 = g["W2"].shape[1]
        return [[G("transform", _gemm_work(V, f_in, F1 + 2 * K)),
                 A("gather", _gather_work(V, E, F1, F1, per_row_bytes=2 * K * 4,
                                          flops_per_edge=2 * F1 + 8 * K))],
                [G("transform", _gemm_work(V, F1, F2 + 2 * K)),
                 A("gather", _gather_work(V, E, F2, F2 // K, per_row_bytes=2 * K * 4,
                                          flops_per_edge=2 * F2 + 8 * K))]]
    if name == "sage_rmat":
        F, Fo = g["W_pool"].shape[0], g["W"].shape[1]
        return [[G("pool transform", _gemm_work(V, F, F)), A("max gather", _gather_work(V, E, F, F)),
                 G("concat transform", _gemm_work(V, 2 * F, Fo))]]
    if name == "gated_rgg":
        F, Fe = g["H"].shape[1], g["E_feat"].shape[1]
        gru_b = (2 * V * F + 2 * F * 3 * F + V * F) * 4
        return [[G("source-gate transform", _gemm_work(V, F, F)),
                 G("destination-gate transform", _gemm_work(V, F, F)),
                 A("gated gather", _gather_work(V, E, F, F, per_edge_bytes=Fe * 4,
                                                per_row_bytes=2 * F * 4,
                                                flops_per_edge=2 * Fe * F + 8 * F)),
                 G("GRU transform", (gru_b, 2 * 2 * V * F * 3 * F))]]
    if name == "sage_lstm":
        F, G4 = g["W_ih"].shape
        H, Fo = G4 // 4, g["W"].shape[1]
        return [[G("input transform", _gemm_work(V, F, G4)),
                 A("LSTM gather", _gather_work(V, E, G4, H, flops_per_edge=2 * H * G4 + 10 * H)),
                 G("concat transform", _gemm_work(V, F + H, Fo))]]
    if name == "rgcn_rmat":
        R, Fi, Fo = g["W_rel"].shape
        pairs, rows = int(rel_counts.pairs), int(rel_counts.pair_rows)
        srcs = min(V, pairs)
        return [[G("relation transform", ((srcs * Fi + R * Fi * Fo + rows * Fo) * 4,
                                          2 * rows * Fi * Fo)),
                 G("self transform", _gemm_work(V, Fi, Fo)),
                 A("typed gather", _gather_work(V, E, Fo, Fo, src_rows=pairs, per_edge_bytes=4,
                                                per_row_bytes=Fo * 4, flops_per_edge=2 * Fo))]]
    raise ValueError(name)


def time_stages(S, torch, model, x, ef, stages, reps, markers=False):
    """Per-repetition ms of every stage of every layer ([layer][stage] lists):
    events recorded by the library after each stage (saga_trace_stages), one
    more before each layer."""
    st = torch.cuda.current_stream()
    evs = []
    for _ in range(reps):
        h = x
        row = []
        for layer, names in zip(model, stages):
            ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(names) + 1)]
            S.saga_trace_stages(ev[1:], markers)
            ev[0].record(st)
            h = layer(h, edge_feat=ef)
            row.append(ev)
        evs.append(row)
    S.saga_trace_stages([])
    torch.cuda.synchronize()
    return [[[evs[r][i][k].elapsed_time(evs[r][i][k + 1]) for r in range(reps)]
             for k in range(len(names))] for i, names in enumerate(stages)]


def suite_rooflines(name, stages, samples):
    """Each stage against its roofline (its mean over the repetitions, with
    median, min and p90): compulsory bytes against 8 TB/s, the transforms'
    flops against the float32 MFMA peak, and, where a counter record in
    profiles/ matches the kernel sources, the measured HBM bytes."""
    out = []
    for li, (layer, tl) in enumerate(zip(stages, samples)):
        for (st, kind, byts, flops), v in zip(layer, tl):
            t_ms = statistics.fmean(v)
            t = t_ms * 1e-3
            d = {"layer": li + 1, "stage": st, "bound": kind, "ms": round(t_ms, 5),
                 "ms_spread": spread(v, 5),
                 "compulsory_bytes": byts, "compulsory_GBps": byts / t / 1e9,
                 "compulsory_frac_of_8TBps": byts / t / PEAK_HBM}
            if kind == "mfma":
                d["TFLOPs"] = flops / t / 1e12
                d["mfma_frac"] = flops / t / PEAK_MFMA["f32"]
            tr = load_traffic(f"suite:{name}:L{li + 1}:{st}", "f32")
            if tr:
                d["counter_GBps"] = tr / t / 1e9
                d["counter_frac_of_8TBps"] = tr / t / PEAK_HBM
            out.append(d)
    return out


def spread(v, nd=4):
    """Median, min and 90th percentile (nearest rank: the ceil(0.9 n)-th
    smallest) of a list of timings."""
    k = max(1, -(-9 * len(v) // 10))
    return {"median": round(statistics.median(v), nd), "min": round(min(v), nd),
            "p90": round(sorted(v)[k - 1], nd)}


def suite(dev, reps=20, oracles=None, schedule=None):
    """Per-workload, per-layer timing of the other six workloads through
    saga_layer (plan built once per graph and timed separately), each layer
    also stage by stage against its roofline; `oracles` (suite_oracles'
    result, taken before the GPU was touched) is reported beside each.
    With `schedule` (a list), the stage loop runs with the library's stage
    markers on and the calls are appended to it (for attributing a counter
    profile's dispatches to stages)."""
    import numpy as np
    import torch

    import paper_2009_00804_amd.layers as LY
    import paper_2009_00804_amd.saga as S
    from synth import configs as Cfg

    out = {}
    for name, desc in SUITE:
        g = Cfg.build(name)
        rp = torch.from_numpy(g["row_ptr"]).to(dev)
        col = torch.from_numpy(g["col_idx"]).to(dev)
        graph = S.Graph(rp, col)
        V, E = g["num_vertices"], g["num_edges"]
        if name == "gcn_er":
            model = LY.gcn2(graph, torch.from_numpy(g["W1"]), torch.from_numpy(g["b1"]),
                            torch.from_numpy(g["W2"]), torch.from_numpy(g["b2"]))
            x, ef = _padded(g["X"][:, :g["dims"][0]], torch, dev), None
        elif name == "gat_ba":
            model, x, ef = LY.gat2(graph, g), _padded(g["X"], torch, dev), None
        elif name == "sage_rmat":
            model, x, ef = LY.sage_pool(graph, g), _padded(g["X"], torch, dev), None
        elif name == "sage_lstm":
            model, x, ef = LY.sage_lstm(graph, g), _padded(g["X"], torch, dev), None
        elif name == "rgcn_rmat":
            et = torch.from_numpy(g["etype"]).to(dev)
            relg = S.RelGraph(graph, et, g["num_rel"])
            model, x, ef = LY.rgcn(graph, relg, g), _padded(g["X"], torch, dev), None
        else:
            model = LY.gated_gru(graph, g)
            x, ef = _padded(g["H"], torch, dev), _padded(g["E_feat"], torch, dev)
        st = torch.cuda.current_stream()
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(len(model) + 1)]
        for _ in range(3):
            LY.run(model, x, edge_feat=ef)
        torch.cuda.synchronize()
        stages = suite_stages(name, g, relg.check() if name == "rgcn_rmat" else None)
        names = [[st_[0] for st_ in layer] for layer in stages]
        stage_samples = time_stages(S, torch, model, x, ef, names, reps, markers=schedule is not None)
        if schedule is not None:
            schedule.append({"workload": name, "layers": names, "calls": reps})
        samples = [[] for _ in model]
        for _ in range(reps):
            h = x
            ev[0].record(st)
            for i, layer in enumerate(model):
                h = layer(h, edge_feat=ef)
                ev[i + 1].record(st)
            torch.cuda.synchronize()
            for i in range(len(model)):
                samples[i].append(ev[i].elapsed_time(ev[i + 1]))
        per = [statistics.fmean(v) for v in samples]
        # plan build alone
        plan_t = []
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        for _ in range(reps):
            e0.record(st)
            S.saga_plan_build(graph.num_dst, graph.num_src, graph.num_edges,
                              C.c_void_p(rp.data_ptr()), C.c_void_p(col.data_ptr()), graph.opts,
                              C.c_void_p(graph.ws.data_ptr()), graph.ws.numel(),
                              S.stream_handle(st))
            e1.record(st)
            torch.cuda.synchronize()
            plan_t.append(e0.elapsed_time(e1))
        out[name] = {
            "workload": desc, "vertices": V, "edges": E,
            "plan_ms": statistics.fmean(plan_t), "plan_ms_spread": spread(plan_t, 5),
            "layers": [{"ms": round(ms, 5), "ms_spread": spread(v, 5),
                        "gteps": E / (ms * 1e-3) / 1e9, "vertices_per_s": V / (ms * 1e-3)}
                       for ms, v in zip(per, samples)],
            "stage_rooflines": suite_rooflines(name, stages, stage_samples)}
        log(f"suite {name}: V={V} E={E} plan {out[name]['plan_ms']:.3f} ms, layers "
            + ", ".join(f"{ms:.3f} ms" for ms in per))
        if name == "rgcn_rmat":
            out[name].update(rgcn_detail(S, torch, graph, relg, model[0], x, g, dev, reps))
            log(f"suite rgcn_rmat: {out[name]['rel_plan_ms']:.3f} ms rel plan, stages "
                + ", ".join(f"{k} {v:.3f}" for k, v in out[name]["stage_ms"].items()))
        if name == "sage_lstm":
            out[name].update(lstm_detail(S, torch, graph, g, x, dev))
            d = out[name]
            log(f"suite sage_lstm: LSTM Gather {d['lstm_gather_ms']:.3f} ms persistent "
                f"({d['lstm_us_per_step_of_longest_row']:.3f} us/step of the longest row), "
                f"{d['degree_traversal_ms']:.3f} ms as {d['degree_traversal_launches']} "
                f"per-degree launches")
        if oracles and name in oracles:
            out[name]["cpu_oracle"] = oracles[name]
        del model, graph
        torch.cuda.empty_cache()
    return out


def lstm_detail(S, torch, graph, g, x, dev, reps=20):
    """The LSTM Gather alone: the single persistent call against the degree
    traversal the paper profiles (Sec. 3.2, Fig. 8b: one launch per distinct
    in-degree, rows of equal degree batched), through saga_lstm_gather_rows
    on the same P = X W_ih + b_ih + b_hh."""
    import ctypes as C

    import numpy as np

    H = g["W_hh"].shape[0]
    V = graph.num_dst
    st = torch.cuda.current_stream()
    sh = S.stream_handle(st)
    P = torch.empty((V, 4 * H), dtype=torch.float32, device=dev)
    Wih = torch.from_numpy(g["W_ih"]).to(dev)
    Whh = torch.from_numpy(g["W_hh"]).to(dev)
    bih = torch.from_numpy(g["b_ih"]).to(dev)
    bhh = torch.from_numpy(g["b_hh"]).to(dev)
    gop = S.saga_gemm_op(S.SAGA_F32, S.SAGA_GEMM_PLAIN, S.SAGA_ACT_NONE, None)
    gws = S.workspace(S.saga_apply_vertex_workspace_size(gop, Wih.shape[0], 0, 4 * H), dev)
    none = S.saga_cmat(None, 0, 0, 0)
    S.saga_apply_vertex(gop, S.cmat(x), S.cmat(Wih), none, none, C.c_void_p(bih.data_ptr()),
                        C.c_void_p(bhh.data_ptr()), S.mat(P), C.c_void_p(gws.data_ptr()), gws.numel(), sh)
    out = torch.empty((V, H), dtype=torch.float32, device=dev)
    ws = S.workspace(S.saga_lstm_gather_workspace_size(graph.plan, H), dev)
    # runs of equal in-degree in the plan's order (d_in descending, id ascending)
    d = np.diff(g["row_ptr"].astype(np.int64))
    ds = np.sort(d)[::-1]
    cuts = np.concatenate([[0], np.flatnonzero(np.diff(ds)) + 1, [V]]).tolist()

    def persistent():
        S.saga_lstm_gather(graph.plan, S.cmat(P), S.cmat(Whh), S.mat(out),
                           C.c_void_p(ws.data_ptr()), ws.numel(), sh)

    def traversal():
        for a, b in zip(cuts[:-1], cuts[1:]):
            S.saga_lstm_gather_rows(graph.plan, a, b, S.cmat(P), S.cmat(Whh), S.mat(out),
                                    C.c_void_p(ws.data_ptr()), ws.numel(), sh)

    res, spr = {}, {}
    st = torch.cuda.current_stream()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for name, f, n in (("persistent", persistent, reps), ("traversal", traversal, 5)):
        f()
        torch.cuda.synchronize()
        v = []
        for _ in range(n):
            e0.record(st)
            f()
            e1.record(st)
            torch.cuda.synchronize()
            v.append(e0.elapsed_time(e1))
        res[name], spr[name] = statistics.fmean(v), spread(v)
    dmax = int(d.max())
    return {"max_in_degree": dmax, "lstm_gather_ms": res["persistent"],
            "lstm_gather_ms_spread": spr["persistent"],
            "lstm_us_per_step_of_longest_row": res["persistent"] * 1e3 / dmax,
            "degree_traversal_ms": res["traversal"], "degree_traversal_launches": len(cuts) - 1,
            "degree_traversal_slowdown": res["traversal"] / res["persistent"]}


def rgcn_detail(S, torch, graph, relg, layer, x, g, dev, reps):
    """R-GCN stage times (typed layout, grouped per-relation transform, self
    GEMM, typed Gather) through the op-level entry points, on the layer's
    own buffers, and the pair counts that size the transform."""
    import ctypes as C

    c = relg.check()
    R, Fi, Fo = g["W_rel"].shape
    rel = relg.rel
    st = torch.cuda.current_stream()
    sh = S.stream_handle(st)
    T = torch.empty((rel.max_pairs, S.gather_ld(Fo, 4)), dtype=torch.float32, device=dev)[:, :Fo]
    SELF = torch.empty((graph.num_dst, S.gather_ld(Fo, 4)), dtype=torch.float32, device=dev)[:, :Fo]
    out = torch.empty_like(SELF)
    Wr = layer.w["w"]
    Ws = layer.w["w_self"]
    b = layer.w["b"]
    tws = S.workspace(S.saga_rel_transform_workspace_size(rel, S.SAGA_F32, Fi, Fo), dev)
    gop = S.saga_gemm_op(S.SAGA_F32, S.SAGA_GEMM_PLAIN, S.SAGA_ACT_NONE, None)
    gws = S.workspace(S.saga_apply_vertex_workspace_size(gop, Fi, 0, Fo), dev)
    op = S.saga_edge_op(S.SAGA_MSG_TYPED, S.SAGA_RED_SUM, S.SAGA_F32, 1, 0, 0, 0.0, S.SAGA_ACT_RELU)
    inp = S.saga_edge_inputs()
    inp.src = S.cmat(T)
    inp.rel = C.pointer(rel)
    inp.self = S.cmat(SELF)
    pws = S.workspace(S.saga_gather_workspace_size(graph.plan, op, Fo), dev)
    none = S.saga_cmat(None, 0, 0, 0)

    def f_plan():
        relg.build()

    def f_transform():
        S.saga_rel_transform(rel, S.SAGA_F32, S.cmat(x), S.cmat(Wr), S.mat(T),
                             C.c_void_p(tws.data_ptr()), tws.numel(), sh)

    def f_self():
        S.saga_apply_vertex(gop, S.cmat(x), S.cmat(Ws), none, none, C.c_void_p(b.data_ptr()), None,
                            S.mat(SELF), C.c_void_p(gws.data_ptr()), gws.numel(), sh)

    def f_gather():
        S.saga_scatter_apply_edge_gather(graph.plan, op, inp, S.mat(out), C.c_void_p(pws.data_ptr()),
                                         pws.numel(), sh)

    res = {}
    for name, f in (("rel_plan", f_plan), ("rel_transform", f_transform), ("self_gemm", f_self),
                    ("typed_gather", f_gather)):
        f()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(reps):
            f()
        e1.record(st)
        torch.cuda.synchronize()
        res[name] = e0.elapsed_time(e1) / reps
    pairs = int(c.pairs)
    E, V = graph.num_edges, graph.num_dst
    return {"rel_plan_ms": res.pop("rel_plan"), "stage_ms": res, "relations": int(R),
            "distinct_pairs": pairs, "pair_rows": int(c.pair_rows),
            "transform_TFLOPs": 2.0 * c.pair_rows * Fi * Fo / (res["rel_transform"] * 1e-3) / 1e12,
            "flops_vs_per_edge": pairs / E,
            "flops_vs_all_relations": pairs / (V * R)}


_CPU_G = None  # the workload, shared with forked baseline workers


def _oracle_rows(g, rows):
    """The oracle's layer-1 GCN (aggregate-first, float64) on some
    destination rows; the degree scalings are computed once, outside."""
    from oracle import saga_oracle as O

    f_in = g["dims"][0]
    rp = g["row_ptr"]
    agg = O.gather(rp, g["col_idx"], g["X"][:, :f_in], "sum", rows=rows, src_scale=g["_s_out"])
    agg = agg * g["_s_in"][rows][:, None]
    O.dense(agg, g["W1"], bias=g["b1"], act="relu")


def _cpu_worker(args):
    seed, budget_s = args
    import numpy as np
    from threadpoolctl import threadpool_limits

    g = _CPU_G
    rp = g["row_ptr"].astype(np.int64)
    rng = np.random.default_rng(seed)
    edges, t, n = 0, 0.0, 0
    with threadpool_limits(1):
        while t < budget_s:
            rows = rng.integers(0, g["num_vertices"], 500)
            t0 = time.perf_counter()
            _oracle_rows(g, rows)
            t += time.perf_counter() - t0
            edges += int((rp[rows + 1] - rp[rows]).sum())
            n += len(rows)
    return edges, n


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(g, budget_s=12.0):
    """The oracle's layer-1 GCN (aggregate-first, float64) on bounded random
    samples of destination rows of the same workload: once on one thread,
    and once on every core of the affinity mask (at most 16), each worker
    process one thread on its own sample.  Runs before the GPU is touched
    (its workers are forked)."""
    import multiprocessing as mp

    import numpy as np

    from oracle import saga_oracle as O

    global _CPU_G
    V = g["num_vertices"]
    g["_s_out"] = O.degree_scale(O.out_degrees(g["col_idx"], V))
    g["_s_in"] = O.degree_scale(np.diff(g["row_ptr"].astype(np.int64)))
    _CPU_G = g
    t0 = time.perf_counter()
    e1, n1 = _cpu_worker((7, budget_s / 2))
    t1 = time.perf_counter() - t0
    cores = max(1, min(len(os.sched_getaffinity(0)), 16))
    en, nn, tn = e1, n1, t1
    if cores > 1:
        t0 = time.perf_counter()
        with mp.get_context("fork").Pool(cores) as pool:
            res = pool.map(_cpu_worker, [(100 + k, budget_s / 2) for k in range(cores)])
        tn = time.perf_counter() - t0
        en, nn = sum(r[0] for r in res), sum(r[1] for r in res)
    _CPU_G = None
    for k in ("_s_out", "_s_in"):
        g.pop(k)
    return dict(value=en / tn, unit="edges/s", cores=cores, kind="oracle", cpu_model=_cpu_model(),
                sample=f"layer-1 GCN (602->128, aggregate-first, float64) on {nn} random destination "
                       f"rows ({en} in-edges) of the same graph, {cores} worker processes of one "
                       f"thread each, {tn:.1f} s wall",
                single_thread={"value": e1 / t1, "unit": "edges/s", "cores": 1,
                               "sample": f"{n1} random destination rows ({e1} in-edges), {t1:.1f} s"})


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--dtype", choices=["f32", "bf16"], default="f32")
    ap.add_argument("--variants", default="bf16", help="extra dtypes to time (comma list or '')")
    ap.add_argument("--scale", type=int, default=21)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--no-suite", action="store_true",
                    help="skip the per-layer timing of the six smaller workloads")
    ap.add_argument("--no-unfused", action="store_true",
                    help="skip the fused-vs-unfused layer-1 aggregation comparison")
    ap.add_argument("--plan-join", choices=["gather", "transform"], default="gather",
                    help="with the pipelined plan, where the step waits for the plan's row-order "
                         "branch: before the first Gather (it overlaps the first transform) or "
                         "before the first transform (it overlaps the out-degree count only); "
                         "both are measured and reported")
    ap.add_argument("--pipeline", choices=["on", "off"], default="on",
                    help="time the step with the plan's row-order branch on a second stream, "
                         "overlapping the first transform (on), or stage by stage (off); both "
                         "are measured and reported")
    ap.add_argument("--fused", choices=["on", "off"], default="off",
                    help="time the step with layer 2's transform fused into layer 1's Gather "
                         "(on) for the headline value; both are measured and reported")
    ap.add_argument("--suite-schedule", default="",
                    help="run the suite's stage loop with the library's stage markers on and "
                         "write its call schedule here (for attributing a counter profile)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="before timing, run one device-to-device copy of this many MiB "
                         "(a known-size kernel for calibrating memory counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the library has no multi-GPU path "
              "(how it would shard is documented, not built); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch

    from synth import configs as Cfg

    t0 = time.time()
    g = Cfg.build("gcn_rmat", scale=args.scale)
    log(f"inputs: V={g['num_vertices']} E={g['num_edges']} in {time.time() - t0:.1f}s")
    cpu = None
    if not args.no_cpu_baseline:
        # before any GPU call: the all-cores leg forks worker processes
        log("cpu baseline (oracle) ...")
        cpu = cpu_baseline(g, args.cpu_budget)
        log(f"cpu baseline: {cpu['value']:.3e} edges/s on {cpu['cores']} cores, "
            f"{cpu['single_thread']['value']:.3e} on one")
    oracles = None
    if not args.no_cpu_baseline and not args.no_suite:
        oracles = suite_oracles()
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    dtypes = [args.dtype] + [d for d in args.variants.split(",") if d and d != args.dtype]
    if "bf16" in dtypes:
        Cfg.add_bf16_variant(g)

    if args.calib_copy_mib:
        n = args.calib_copy_mib << 18
        a = torch.ones(n, dtype=torch.float32, device=dev)
        b = torch.empty_like(a)
        b.copy_(a)
        torch.cuda.synchronize()
        log(f"calibration copy: {args.calib_copy_mib} MiB")
        del a, b
    results = {}
    for dt in dtypes:
        step = Step(g, dt, dev)
        counts = step.graph.counts
        # stage-by-stage first (per-stage times are attributed cleanly), then
        # with the plan's row order overlapping the first transform
        wall, per, tot = time_step(step, args.steps, args.warmup)
        ms_seq = wall * 1e3 / args.steps
        med = {n: statistics.median(v) for n, v in per.items()}
        mean = {n: statistics.fmean(v) for n, v in per.items()}
        # per stage over the timed steps: median, min and 90th percentile
        stage_spread = {n: spread(v) for n, v in per.items()}
        step.split = True
        wall_p, _, _ = time_step(step, args.steps, args.warmup)
        ms_pipe = wall_p * 1e3 / args.steps
        # the plan's two branches joined before the transform instead
        step.join_early = True
        wall_j, _, _ = time_step(step, args.steps, args.warmup)
        ms_pipe_early = wall_j * 1e3 / args.steps
        step.join_early = args.plan_join == "transform"
        if step.join_early:
            ms_pipe_late, ms_pipe = ms_pipe, ms_pipe_early
        else:
            ms_pipe_late = ms_pipe
        # and with layer 2's transform fused into layer 1's Gather
        step.fused = True
        wall_f, per_f, _ = time_step(step, args.steps, args.warmup)
        ms_fused = wall_f * 1e3 / args.steps
        fused_gather1 = statistics.fmean(per_f["gather1"])
        step.split = args.pipeline == "on"
        step.fused = args.fused == "on"
        ms = ms_fused if step.fused else (ms_pipe if step.split else ms_seq)
        results[dt] = dict(step=step, ms=ms, med=med, mean=mean, spread=stage_spread, counts=counts,
                           ev_ms=statistics.median(tot), ms_seq=ms_seq, ms_pipe=ms_pipe,
                           ms_fused=ms_fused, fused_gather1=fused_gather1,
                           ms_pipe_early=ms_pipe_early, ms_pipe_late=ms_pipe_late)
        log(f"{dt}: {ms_seq:.3f} ms/step stage by stage (events {statistics.median(tot):.3f}); "
            + ", ".join(f"{n} {med[n]:.3f}" for n in step.names)
            + f"; {ms_pipe:.3f} ms/step with the plan's row order overlapping gemm1"
            + f"; {ms_fused:.3f} ms/step with layer 2's transform fused into layer 1's Gather "
              f"({fused_gather1:.3f} ms for the fused stage)")
        if not args.no_unfused:
            um = time_unfused(step)
            results[dt]["unfused_ms"] = um
            log(f"{dt}: layer-1 aggregation unfused {um:.3f} ms vs fused {mean['gather1']:.3f} ms")
        if dt != args.dtype:
            del step
            results[dt]["step"] = None
            torch.cuda.empty_cache()

    r = results[args.dtype]
    step = r["step"]
    E, V = step.E, step.V
    value = 2 * E / (r["ms"] * 1e-3)
    # dominant kernel of the step
    stages = ["gemm1", "gather1", "gemm2", "gather2"]
    dom = max(stages, key=lambda n: r["mean"][n])
    byts, flops = algorithmic(step, dom)
    dur = r["mean"][dom] * 1e-3
    kernel_name = {"gather1": "k_gather_sum", "gather2": "k_gather_sum",
                   "gemm1": "k_gemm_bres" if args.dtype == "bf16" else "k_gemm",
                   "gemm2": "k_gemm"}[dom]
    if dom.startswith("gemm") and args.dtype == "f32":
        roof = dict(bound="mfma", achieved=flops / dur / 1e12, peak=PEAK_MFMA["f32"] / 1e12,
                    unit="TFLOP/s")
    else:
        roof = dict(bound="hbm", achieved=byts / dur / 1e9, peak=PEAK_HBM / 1e9, unit="GB/s")
    roof["frac"] = roof["achieved"] / roof["peak"]
    roof["traffic"] = load_traffic(f"{dom}", args.dtype)
    roof["kernel"] = f"{dom} ({kernel_name})"
    roof["launch_ms"] = r["mean"][dom]
    roof["algorithmic_bytes"] = byts
    roof["algorithmic"] = ("compulsory bytes: 4 B per CSR index + row_ptr + source matrix "
                           "and output once" if roof["bound"] == "hbm" else "2 M K N flops")
    if roof["traffic"]:
        # measured HBM traffic (rocprofv3 FETCH_SIZE + WRITE_SIZE, calibrated)
        roof["counter_GBps"] = roof["traffic"] / dur / 1e9
        roof["counter_frac_of_8TBps"] = roof["counter_GBps"] / (PEAK_HBM / 1e9)
        roof["traffic_note"] = ("FETCH_SIZE counts L2 egress, Infinity Cache hits included: an "
                                "upper bound on DRAM bytes")
    stage_ms = {n: round(r["mean"][n], 4) for n in step.names}
    out = {
        "metric": "GNN layer throughput: edges/s (GTEPS) + achieved HBM GB/s fraction, 1 MI355X",
        "value": value,
        "unit": "edges/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": r["ms"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.dtype,
        "data": "synthetic (seeded R-MAT + N(0,1) features, random-init Glorot weights)",
        "config": {"workload": "2-layer GCN, R-MAT scale 21 (a,b,c=0.57,0.19,0.19), 50 edges/vertex "
                               "+ self-loops, features 602->128->41",
                   "vertices": V, "edges": E, "layers": 2, "parallelism": "single GPU"},
        "gteps": value / 1e9,
        "vertices_per_s": 2 * V / (r["ms"] * 1e-3),
        "stage_ms": stage_ms,
        "stage_ms_spread": r["spread"],
        "gather1_noreuse_GBps": noreuse_bytes(step, "gather1") / (r["mean"]["gather1"] * 1e-3) / 1e9,
        "gemm1_TFLOPs": algorithmic(step, "gemm1")[1] / (r["mean"]["gemm1"] * 1e-3) / 1e12,
        "plan": {"segments": r["counts"].num_segments, "blocks": r["counts"].num_blocks,
                 "split_rows": r["counts"].n_split, "max_in_degree": r["counts"].max_in_degree},
        "roofline": roof,
        "stage_rooflines": stage_rooflines(V, E, step.dims, args.dtype, r["mean"]),
    }
    out["pipelining"] = {
        "what": "plan's row-order branch (in-degrees, validation, degree sort, segments, "
                "blocks) on a second stream, overlapping the d_out-scaled layer-1 transform",
        "stage_by_stage_ms": r["ms_seq"], "pipelined_ms": r["ms_pipe"],
        "speedup": r["ms_seq"] / r["ms_pipe"], "value_uses": args.pipeline,
        "joined_before_gather_ms": r["ms_pipe_late"],
        "joined_before_transform_ms": r["ms_pipe_early"], "join": args.plan_join}
    out["cross_stage_fusion"] = {
        "what": "layer 2's transform (d_out^-1/2 (h1 W2)) done inside layer 1's last Gather "
                "pass, each wave multiplying the rows it has just finished on the matrix cores "
                "(saga_scatter_apply_edge_gather_transform), instead of a separate GEMM over "
                "all rows after the Gather; with the plan's row order overlapping gemm1",
        "pipelined_ms": r["ms_pipe"], "fused_ms": r["ms_fused"],
        "unfused_gather1_plus_gemm2_ms": r["mean"]["gather1"] + r["mean"]["gemm2"],
        "fused_stage_ms": r["fused_gather1"], "speedup": r["ms_pipe"] / r["ms_fused"],
        "value_uses": args.fused}
    if "unfused_ms" in r:
        out["fusion"] = {
            "stage": "layer-1 Scatter+ApplyEdge+Gather (Fig. 7a unfused vs Fig. 7b fused)",
            "fused_ms": r["mean"]["gather1"], "unfused_ms": r["unfused_ms"],
            "speedup": r["unfused_ms"] / r["mean"]["gather1"]}
    for dt in dtypes[1:]:
        rr = results[dt]
        out.setdefault("variants", {})[dt] = {
            "value": 2 * E / (rr["ms"] * 1e-3), "ms_per_step": rr["ms"],
            "stage_by_stage_ms": rr["ms_seq"], "pipelined_ms": rr["ms_pipe"],
            "joined_before_gather_ms": rr["ms_pipe_late"],
            "joined_before_transform_ms": rr["ms_pipe_early"],
            "fused_ms": rr["ms_fused"], "fused_stage_ms": rr["fused_gather1"],
            "stage_ms": {n: round(rr["mean"][n], 4) for n in rr["mean"]},
            "stage_ms_spread": rr["spread"],
            "stage_rooflines": stage_rooflines(V, E, step.dims, dt, rr["mean"])}
        if "unfused_ms" in rr:
            out["variants"][dt]["fusion"] = {"fused_ms": rr["mean"]["gather1"],
                                             "unfused_ms": rr["unfused_ms"],
                                             "speedup": rr["unfused_ms"] / rr["mean"]["gather1"]}
    if not args.no_suite:
        schedule = [] if args.suite_schedule else None
        out["suite"] = suite(dev, oracles=oracles, schedule=schedule)
        if schedule is not None:
            with open(args.suite_schedule, "w") as f:
                json.dump(schedule, f)
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
