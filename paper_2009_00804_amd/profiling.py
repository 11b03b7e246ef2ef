"""Summaries of rocprofv3 output for the benchmark workload.

Turns the CSV output of three rocprofv3 runs of ``bench.py`` into short text
summaries and a machine-readable per-launch traffic record:

  kernel trace : rocprofv3 --kernel-trace --stats -f csv -- python3 bench.py ...
  FETCH_SIZE   : rocprofv3 --pmc FETCH_SIZE -f csv -- python3 bench.py ... --calib-copy-mib N
  WRITE_SIZE   : rocprofv3 --pmc WRITE_SIZE -f csv -- python3 bench.py ... --calib-copy-mib N

The counter values (KiB per dispatch) are scaled by what the same counter
reads for the known-size device copy that ``--calib-copy-mib`` runs: the
factor is true bytes / counted bytes.

Usage:
  python -m paper_2009_00804_amd.profiling --trace DIR --fetch DIR --write DIR \\
      --copy-mib 1024 --dtype f32 --command "..." --out profiles

Counter mode: any other --pmc passes of the same bench.py command,
summarised per stage with derived figures (L2 hit rate, L1->L2 latency and
reads in flight, MFMA busy):
  python -m paper_2009_00804_amd.profiling --counters DIR1,DIR2 --dtype f32 \\
      --command "..." --passes "..." --out profiles

Suite mode (the other workloads, stage by stage): bench.py run with
``--suite-schedule FILE`` launches the library's stage markers
(k_stage_begin, k_stage_mark) around every stage of its traced layer calls
and writes the order of those calls to FILE; ``--suite FILE`` then
attributes every dispatch of the FETCH_SIZE and WRITE_SIZE runs to its
workload, layer and stage:
  python -m paper_2009_00804_amd.profiling --suite FILE --fetch DIR --write DIR \\
      --copy-mib 1024 --command "..." --out profiles

Marker mode (a rocprofv3 --marker-trace run of the same bench.py command):
the roctx ranges saga_layer opens ("saga_layer", "saga stage k") are
checked against the schedule and summarised per layer call and stage:
  python -m paper_2009_00804_amd.profiling --suite FILE --markers DIR \\
      --command "..." --out profiles
"""
from __future__ import annotations

import argparse
import collections
import csv
import glob
import hashlib
import json
import os
import re

PKG = os.path.dirname(os.path.abspath(__file__))

# stage -> ({dtype: [(kernel-name prefix, dispatches per launch, cycle,
# slots), ...]}, source file).  A kernel that several stages of one step
# launch (the same instance serves the layer-1 slices and the layer-2
# whole-line pass) is split by position: of every `cycle` consecutive
# dispatches of it, the stage takes those at `slots`.  gather1 runs one
# dispatch per 128-byte column slice; the float32 gather2 runs the 32
# whole-line columns and the 9-column rest; each Gather with split rows ends
# with a combine.
STAGES = {
    # the plan's out-degree count (tile sort by bucket, per-bucket count,
    # partial sums), once per step
    "outdeg": ({dt: [("k_outdeg_bin", 1, 1, (0,)), ("k_outdeg_count", 1, 1, (0,)),
                     ("k_outdeg_reduce", 1, 1, (0,))] for dt in ("f32", "bf16")},
               "plan.hip"),
    "gather1": ({"f32": [("k_gather_sum<float, 8, 1, 4, 4, true>", 4, 5, (0, 1, 2, 3)),
                         ("k_combine<float>", 1, 3, (0,))],
                 "bf16": [("k_gather_sum<unsigned short, 8, 1, 4, 4, true>", 2, 2, (0, 1)),
                          ("k_combine<unsigned short>", 1, 2, (0,))]},
                "gather.hip"),
    "gather2": ({"f32": [("k_gather_sum<float, 8, 1, 4, 4, true>", 1, 5, (4,)),
                         ("k_gather_sum<float, 4, 1, 4, 8, false>", 1, 1, (0,)),
                         ("k_combine<float>", 2, 3, (1, 2))],
                 "bf16": [("k_gather_sum<unsigned short, 8, 1, 4, 4, false>", 1, 1, (0,)),
                          ("k_combine<unsigned short>", 1, 2, (1,))]},
                "gather.hip"),
    "gemm1": ({"f32": [("k_gemm<float, 2, 8,", 1, 1, (0,))],
               "bf16": [("k_gemm_bres<2, 8, 3>", 1, 1, (0,))]},
              "gemm.hip"),
    "gemm2": ({"f32": [("k_gemm<float, 2, 3,", 1, 1, (0,))],
               "bf16": [("k_gemm<unsigned short, 2, 3,", 1, 1, (0,))]},
              "gemm.hip"),
}


def _short(name):
    name = name.replace("void saga::(anonymous namespace)::", "")
    name = name.replace("saga::(anonymous namespace)::", "")
    name = name.replace("(anonymous namespace)::", "")
    return re.sub(r"\((saga::|int|long|unsigned).*$", "", name)


def _csv(d, suffix):
    hits = glob.glob(os.path.join(d, "**", f"*{suffix}"), recursive=True)
    if not hits:
        raise FileNotFoundError(f"no *{suffix} under {d}")
    return hits[0]


def src_sha(name):
    with open(os.path.join(PKG, "csrc", name), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def kernel_stats(trace_dir):
    """{short kernel name: (calls, avg_us, total_us, min_us, max_us)} from
    the kernel trace."""
    rows = list(csv.DictReader(open(_csv(trace_dir, "kernel_trace.csv"))))
    acc = collections.defaultdict(list)
    for r in rows:
        acc[_short(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    return {k: (len(v), sum(v) / len(v), sum(v), min(v), max(v)) for k, v in acc.items()}


def trace_lists(trace_dir):
    """{short kernel name: [duration us, ...]} in dispatch order."""
    rows = list(csv.DictReader(open(_csv(trace_dir, "kernel_trace.csv"))))
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    acc = collections.defaultdict(list)
    for r in rows:
        acc[_short(r["Kernel_Name"])].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    return acc


def counter_avgs(counter_dir, counter):
    rows = list(csv.DictReader(open(_csv(counter_dir, "counter_collection.csv"))))
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    acc = collections.defaultdict(list)
    for r in rows:
        if r["Counter_Name"] == counter:
            acc[_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return acc


def calibration(acc, copy_mib):
    """true bytes / counted bytes for the known-size copy (largest dispatch
    of the runtime's copy kernel)."""
    vals = acc.get("__amd_rocclr_copyBuffer") or []
    if not vals:
        return None
    counted_kib = max(vals)
    return (copy_mib * 1024.0) / counted_kib if counted_kib > 0 else None


# main kernel source of each suite stage (the traffic record is valid while
# its hash matches)
def _stage_source(stage):
    if stage == "LSTM gather":
        return "lstm.hip"
    return "gather.hip" if "gather" in stage else "gemm.hip"


def dispatches(counter_dir, counter):
    """[(kernel name, value)] in dispatch order."""
    rows = [r for r in csv.DictReader(open(_csv(counter_dir, "counter_collection.csv")))
            if r["Counter_Name"] == counter]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    return [(_short(r["Kernel_Name"]), float(r["Counter_Value"])) for r in rows]


def attribute(disp, schedule):
    """Sum of each (workload, layer, stage)'s counter values over the traced
    calls, and the kernels seen in each, walking the dispatches between the
    stage markers in the order the schedule lists the calls."""
    calls = []
    for w in schedule:
        for _ in range(w["calls"]):
            for li, stages in enumerate(w["layers"]):
                calls.append((w["workload"], li + 1, stages))
    acc, kern = collections.defaultdict(float), collections.defaultdict(set)
    ci, stage, inside = 0, 0, False
    for name, val in disp:
        if name.startswith("k_stage_begin"):
            if ci >= len(calls):
                raise ValueError("more traced calls in the profile than in the schedule")
            inside, stage = True, 0
            continue
        if not inside:
            continue
        wl, li, stages = calls[ci]
        if name.startswith("k_stage_mark"):
            stage += 1
            if stage == len(stages):
                inside = False
                ci += 1
            continue
        acc[(wl, li, stages[stage])] += val
        kern[(wl, li, stages[stage])].add(name)
    if ci != len(calls):
        raise ValueError(f"profile holds {ci} traced calls, the schedule {len(calls)}")
    return acc, kern


def marker_ranges(marker_dir):
    """[(name, start ns, end ns)] of the roctx ranges of a --marker-trace
    run, by start time (an enclosing range before the ranges it holds)."""
    rows = csv.DictReader(open(_csv(marker_dir, "marker_api_trace.csv")))
    out = [(r["Function"], int(r["Start_Timestamp"]), int(r["End_Timestamp"])) for r in rows]
    out.sort(key=lambda x: (x[1], -x[2]))
    return out


def attribute_ranges(ranges, schedule):
    """Host time (ns) of every traced layer call and of each of its stages,
    walking the "saga_layer" ranges in the order the schedule lists the
    calls.  Each layer range must hold its stages' ranges "saga stage 0"
    .. "saga stage n-1", in order and nested inside it; anything else
    raises ValueError.  Returns ({(workload, layer): [ns]},
    {(workload, layer, stage): [ns]})."""
    calls = []
    for w in schedule:
        for _ in range(w["calls"]):
            for li, stages in enumerate(w["layers"]):
                calls.append((w["workload"], li + 1, stages))
    layers = [r for r in ranges if r[0] == "saga_layer"]
    stage_r = [r for r in ranges if r[0].startswith("saga stage ")]
    if len(layers) != len(calls):
        raise ValueError(f"trace holds {len(layers)} layer ranges, the schedule {len(calls)} calls")
    lay, acc = collections.defaultdict(list), collections.defaultdict(list)
    si = 0
    for (wl, li, names), (_, t0, t1) in zip(calls, layers):
        lay[(wl, li)].append(t1 - t0)
        for k, nm in enumerate(names):
            if si >= len(stage_r):
                raise ValueError("fewer stage ranges than the schedule's stages")
            rn, s0, s1 = stage_r[si]
            if rn != f"saga stage {k}" or s0 < t0 or s1 > t1:
                raise ValueError(f"range {si} ({rn}) is not stage {k} of its layer call")
            acc[(wl, li, nm)].append(s1 - s0)
            si += 1
    if si != len(stage_r):
        raise ValueError(f"{len(stage_r) - si} stage ranges outside the traced calls")
    return lay, acc


def markers_main(a):
    """Summary of the roctx ranges ("saga_layer", "saga stage k") of a
    --marker-trace run of the suite: host time per layer call and stage."""
    schedule = json.load(open(a.suite))
    lay, acc = attribute_ranges(marker_ranges(a.markers), schedule)
    med = lambda v: sorted(v)[(len(v) - 1) // 2] / 1e3  # noqa: E731
    lines = ["# roctx ranges of the traced saga_layer calls: the suite workloads (float32)", "",
             f"command: {a.command}",
             "summary: python -m paper_2009_00804_amd.profiling --suite OUT/schedule.json "
             "--markers OUT --command '...' --out profiles", "",
             "Each layer call is one \"saga_layer\" range holding one \"saga stage k\" range per",
             "stage, in order; every range was checked against the call schedule. The ranges",
             "bracket the host side of each call (argument checks and kernel enqueue; the GPU",
             "work runs asynchronously). Host microseconds, median and max over the calls; the",
             "run traces markers only (a kernel trace adds a per-dispatch cost to these times).", "",
             f"{'workload':10s} {'layer':>5s} {'stage':28s} {'calls':>6s} {'median us':>10s} "
             f"{'max us':>10s}"]
    for w in schedule:
        for li, stages in enumerate(w["layers"]):
            v = lay[(w["workload"], li + 1)]
            lines.append(f"{w['workload']:10s} {li + 1:5d} {'(whole call)':28s} {len(v):6d} "
                         f"{med(v):10.1f} {max(v) / 1e3:10.1f}")
            for st in stages:
                v = acc[(w["workload"], li + 1, st)]
                lines.append(f"{'':10s} {'':5s} {st:28s} {len(v):6d} {med(v):10.1f} "
                             f"{max(v) / 1e3:10.1f}")
    with open(os.path.join(a.out, "marker_ranges_suite_f32.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")


def suite_main(a):
    schedule = json.load(open(a.suite))
    fe, wr = dispatches(a.fetch, "FETCH_SIZE"), dispatches(a.write, "WRITE_SIZE")
    cf = calibration({"__amd_rocclr_copyBuffer": [v for n, v in fe if n == "__amd_rocclr_copyBuffer"]},
                     a.copy_mib)
    cw = calibration({"__amd_rocclr_copyBuffer": [v for n, v in wr if n == "__amd_rocclr_copyBuffer"]},
                     a.copy_mib)
    fa, fk = attribute(fe, schedule)
    wa, _ = attribute(wr, schedule)
    ncalls = {w["workload"]: w["calls"] for w in schedule}
    lines = ["# HBM traffic per stage: the suite workloads (float32)", "",
             f"command (FETCH_SIZE pass): {a.command} --pmc FETCH_SIZE",
             f"command (WRITE_SIZE pass): {a.command} --pmc WRITE_SIZE", "",
             f"calibration copy: {a.copy_mib:.0f} MiB device-to-device; FETCH_SIZE scale "
             f"{cf:.3f}, WRITE_SIZE scale {cw:.3f} (true bytes / counted bytes)", "",
             f"{'workload':10s} {'layer':>5s} {'stage':28s} {'FETCH MB':>10s} {'WRITE MB':>10s}  kernels"]
    rec_path = os.path.join(a.out, "traffic.json")
    rec = json.load(open(rec_path)) if os.path.exists(rec_path) else {}
    for key in sorted(fa, key=lambda k: (k[0], k[1])):
        wl, li, stage = key
        n = ncalls[wl]
        fb = fa[key] * cf * 1024 / n
        wb = wa.get(key, 0.0) * cw * 1024 / n
        lines.append(f"{wl:10s} {li:5d} {stage:28s} {fb / 1e6:10.2f} {wb / 1e6:10.2f}  "
                     + ", ".join(sorted(k[:48] for k in fk[key])))
        src = _stage_source(stage)
        rec[f"suite:{wl}:L{li}:{stage}:f32"] = {
            "kernels": sorted(fk[key]), "source": src, "src_sha": src_sha(src),
            "bytes_per_launch": fb + wb, "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
            "calibration": {"fetch": cf, "write": cw}}
    with open(os.path.join(a.out, "hbm_traffic_suite_f32.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")
    with open(rec_path, "w") as f:
        json.dump(rec, f, indent=1, sort_keys=True)


def all_counter_lists(counter_dir):
    """{counter: {short kernel name: [value per dispatch, ...]}} in dispatch
    order, every counter of one --pmc pass."""
    rows = list(csv.DictReader(open(_csv(counter_dir, "counter_collection.csv"))))
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    acc = collections.defaultdict(lambda: collections.defaultdict(list))
    for r in rows:
        acc[r["Counter_Name"]][_short(r["Kernel_Name"])].append(float(r["Counter_Value"]))
    return acc


# derived figures of a stage from its per-launch counter sums: (label,
# numerator, denominator terms, scale).  GRBM_GUI_ACTIVE reads the sum over
# the 8 XCDs (8 x the kernel's cycles: about 8.5e7 for a 4.7 ms launch at
# 2.4 GHz), the TCP counters the sum over the 256 CUs' L1s and
# SQ_VALU_MFMA_BUSY_CYCLES the sum over the 1,024 SIMDs, so "per CU" divides
# by 256 x GRBM_GUI_ACTIVE / 8 and "per SIMD" by 1,024 x GRBM_GUI_ACTIVE / 8.
NUM_XCD, NUM_CU, NUM_SIMD = 8, 256, 1024
DERIVED = [
    ("L2 hit rate", "TCC_HIT_sum", ("TCC_HIT_sum", "TCC_MISS_sum"), 1.0),
    ("L1->L2 read latency, cycles per request", "TCP_TCC_READ_REQ_LATENCY_sum",
     ("TCP_TCC_READ_REQ_sum",), 1.0),
    ("L1->L2 reads in flight per CU", "TCP_TCC_READ_REQ_LATENCY_sum", ("GRBM_GUI_ACTIVE",),
     NUM_XCD / NUM_CU),
    ("fraction of CU cycles with L1 misses pending (stalled)", "TCP_PENDING_STALL_CYCLES_sum",
     ("GRBM_GUI_ACTIVE",), NUM_XCD / NUM_CU),
    ("MFMA busy fraction per SIMD", "SQ_VALU_MFMA_BUSY_CYCLES", ("GRBM_GUI_ACTIVE",),
     NUM_XCD / NUM_SIMD),
    ("LDS bank conflicts per LDS instruction", "SQ_LDS_BANK_CONFLICT", ("SQ_INSTS_LDS",), 1.0),
]


def counters_main(a):
    """Per-stage counter summary of --pmc passes over the benchmark step."""
    per_stage = collections.defaultdict(dict)
    names = []
    for d in a.counters.split(","):
        for cname, by_kernel in all_counter_lists(d).items():
            if cname in names:
                continue
            names.append(cname)
            for stage, (pats, _src) in STAGES.items():
                total, ok = 0.0, True
                for pat, per, cycle, slots in pats[a.dtype]:
                    keys = [k for k in by_kernel if k.startswith(pat)]
                    if len(keys) != 1:
                        ok = False
                        break
                    v = [x for i, x in enumerate(by_kernel[keys[0]]) if i % cycle in slots]
                    if not v:
                        ok = False
                        break
                    total += per * sum(v) / len(v)
                if ok:
                    per_stage[stage][cname] = total
    lines = [f"# Counters per stage launch: {a.tag} ({a.dtype})", "",
             f"command: {a.command} (one run per pass; passes: {a.passes})", "",
             "Each value is the counter's per-dispatch average over the run, summed over",
             "the dispatches one launch of the stage makes (the kernel-to-stage rules",
             "are profiling.STAGES).", ""]
    for stage in STAGES:
        if stage not in per_stage:
            continue
        c = per_stage[stage]
        lines.append(f"## {stage}")
        for cname in names:
            if cname in c:
                lines.append(f"  {cname:36s} {c[cname]:16.4g}")
        for label, num, den, scale in DERIVED:
            if num in c and all(d in c for d in den):
                dv = sum(c[d] for d in den)
                if dv > 0:
                    lines.append(f"  = {label}: {scale * c[num] / dv:.4g}")
        lines.append("")
    with open(os.path.join(a.out, f"counters_{a.tag}_{a.dtype}.txt"), "w") as f:
        f.write("\n".join(lines))


def suite_counters_main(a):
    """Per-stage counter summary of --pmc passes over the suite's traced
    layer calls (stage markers on), with the derived figures of DERIVED."""
    schedule = json.load(open(a.suite))
    ncalls = {w["workload"]: w["calls"] for w in schedule}
    per, kern, names = collections.defaultdict(dict), {}, []
    for d in a.counters.split(","):
        for cname in sorted(all_counter_lists(d)):
            if cname in names:
                continue
            names.append(cname)
            acc, k = attribute(dispatches(d, cname), schedule)
            for key, v in acc.items():
                per[key][cname] = v / ncalls[key[0]]
                kern.setdefault(key, k[key])
    order = [w["workload"] for w in schedule]
    lines = ["# Counters per stage: the suite workloads (float32)", "",
             f"command: {a.command} (one run per pass; passes: {a.passes})", "",
             "Each value is the stage's counter total over one layer call (the sum over",
             "the dispatches between the library's stage markers, averaged over the",
             "traced calls); derived figures as in the benchmark step's summary.", ""]
    for key in sorted(per, key=lambda k: (order.index(k[0]), k[1])):
        wl, li, stage = key
        c = per[key]
        lines.append(f"## {wl} layer {li}: {stage}  ({', '.join(sorted(x[:40] for x in kern[key]))})")
        for cname in names:
            if cname in c:
                lines.append(f"  {cname:36s} {c[cname]:16.4g}")
        for label, num, den, scale in DERIVED:
            if num in c and all(x in c for x in den):
                dv = sum(c[x] for x in den)
                if dv > 0:
                    lines.append(f"  = {label}: {scale * c[num] / dv:.4g}")
        lines.append("")
    with open(os.path.join(a.out, "counters_suite_f32.txt"), "w") as f:
        f.write("\n".join(lines))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace")
    ap.add_argument("--suite", help="call schedule written by bench.py --suite-schedule")
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-mib", type=float, default=1024)
    ap.add_argument("--dtype", default="f32")
    ap.add_argument("--command", default="")
    ap.add_argument("--out", default="profiles")
    ap.add_argument("--tag", default="gcn_rmat21")
    ap.add_argument("--counters", help="comma-separated --pmc output directories (counter mode)")
    ap.add_argument("--passes", default="", help="the counters of each pass, for the header")
    ap.add_argument("--markers", help="--marker-trace output directory (with --suite: range mode)")
    a = ap.parse_args()
    os.makedirs(a.out, exist_ok=True)
    if a.suite and a.markers:
        return markers_main(a)
    if a.suite:
        return suite_counters_main(a) if a.counters else suite_main(a)
    if a.counters:
        return counters_main(a)

    st = kernel_stats(a.trace)
    tot = sum(v[2] for v in st.values())
    lines = [f"# Kernel trace summary: {a.tag} ({a.dtype})", "",
             f"command: {a.command}", "",
             f"{'kernel':70s} {'calls':>6s} {'avg us':>10s} {'min us':>10s} {'max us':>10s} "
             f"{'% time':>7s}"]
    for k, (n, avg, total, lo, hi) in sorted(st.items(), key=lambda kv: -kv[1][2]):
        lines.append(f"{k[:70]:70s} {n:6d} {avg:10.1f} {lo:10.1f} {hi:10.1f} {100 * total / tot:7.2f}")
    with open(os.path.join(a.out, f"kernel_trace_{a.tag}_{a.dtype}.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")

    if not (a.fetch and a.write):
        return
    fe = counter_avgs(a.fetch, "FETCH_SIZE")
    wr = counter_avgs(a.write, "WRITE_SIZE")
    cf, cw = calibration(fe, a.copy_mib), calibration(wr, a.copy_mib)
    lines = [f"# HBM traffic per dispatch: {a.tag} ({a.dtype})", "",
             f"command (FETCH_SIZE pass): {a.command} --pmc FETCH_SIZE",
             f"command (WRITE_SIZE pass): {a.command} --pmc WRITE_SIZE", "",
             f"calibration copy: {a.copy_mib:.0f} MiB device-to-device; FETCH_SIZE scale "
             f"{cf:.3f}, WRITE_SIZE scale {cw:.3f} (true bytes / counted bytes)", "",
             f"{'kernel':70s} {'FETCH KiB':>12s} {'WRITE KiB':>12s} {'GB (scaled)':>12s}"]
    for k in sorted(set(fe) | set(wr)):
        f_ = sum(fe.get(k, [0])) / max(1, len(fe.get(k, [0])))
        w_ = sum(wr.get(k, [0])) / max(1, len(wr.get(k, [0])))
        gb = (f_ * cf + w_ * cw) * 1024 / 1e9
        lines.append(f"{k[:70]:70s} {f_:12.0f} {w_:12.0f} {gb:12.3f}")
    with open(os.path.join(a.out, f"hbm_traffic_{a.tag}_{a.dtype}.txt"), "w") as f:
        f.write("\n".join(lines) + "\n")

    rec_path = os.path.join(a.out, "traffic.json")
    rec = json.load(open(rec_path)) if os.path.exists(rec_path) else {}
    tr_us = trace_lists(a.trace)
    for stage, (pats, src) in STAGES.items():
        parts = []
        for pat, per, cycle, slots in pats[a.dtype]:
            keys = [k for k in set(fe) | set(wr) if k.startswith(pat)]
            if len(keys) != 1:
                break
            parts.append((keys[0], per, cycle, slots))
        if len(parts) != len(pats[a.dtype]):
            continue
        entry = {"kernels": [], "source": src, "src_sha": src_sha(src), "bytes_per_launch": 0.0,
                 "trace_us_per_launch": 0.0, "calibration": {"fetch": cf, "write": cw}}
        for k, per, cycle, slots in parts:
            pick = lambda v: [x for i, x in enumerate(v) if i % cycle in slots] or [0.0]  # noqa: E731
            f_ = sum(pick(fe[k])) / len(pick(fe[k]))
            w_ = sum(pick(wr[k])) / len(pick(wr[k]))
            n_avg = sum(pick(tr_us.get(k, []))) / len(pick(tr_us.get(k, [])))
            entry["kernels"].append({
                "kernel": k, "dispatches_per_launch": per,
                "fetch_bytes_per_dispatch": f_ * cf * 1024,
                "write_bytes_per_dispatch": w_ * cw * 1024, "trace_avg_us_per_dispatch": n_avg})
            entry["bytes_per_launch"] += per * (f_ * cf + w_ * cw) * 1024
            entry["trace_us_per_launch"] += per * n_avg
        rec[f"{stage}:{a.dtype}"] = entry
    with open(rec_path, "w") as f:
        json.dump(rec, f, indent=1, sort_keys=True)


if __name__ == "__main__":
    main()
