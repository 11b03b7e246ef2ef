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

# stage -> ({dtype: [(kernel-name prefix, dispatches per launch), ...]}, source file).
# gather1 runs one dispatch per 128-byte column slice; the float32 gather2
# runs two kernels (the 32 whole-line columns and the 9-column rest).
STAGES = {
    "gather1": ({"f32": [("k_gather_simple<float, 8, 1, 8, 4, false, 0, true", 4)],
                 "bf16": [("k_gather_simple<unsigned short, 8, 1, 8, 4, false, 0, true", 2)]},
                "gather.hip"),
    "gather2": ({"f32": [("k_gather_simple<float, 8, 1, 8, 4, false, 0, false", 1),
                         ("k_gather_simple<float, 4, 1, 4, 8, false, 0, false", 1)],
                 "bf16": [("k_gather_simple<unsigned short, 8, 1, 8, 4, false, 0, false", 1)]},
                "gather.hip"),
    "gemm1": ({"f32": [("k_gemm<float, 2, 8,", 1)], "bf16": [("k_gemm_bres<2, 8, 3>", 1)]},
              "gemm.hip"),
    "gemm2": ({"f32": [("k_gemm<float, 2, 3,", 1)], "bf16": [("k_gemm<unsigned short, 2, 3,", 1)]},
              "gemm.hip"),
}


def _short(name):
    name = name.replace("void saga::(anonymous namespace)::", "")
    name = name.replace("saga::(anonymous namespace)::", "")
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


def counter_avgs(counter_dir, counter):
    rows = list(csv.DictReader(open(_csv(counter_dir, "counter_collection.csv"))))
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


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--trace", required=True)
    ap.add_argument("--fetch")
    ap.add_argument("--write")
    ap.add_argument("--copy-mib", type=float, default=1024)
    ap.add_argument("--dtype", default="f32")
    ap.add_argument("--command", default="")
    ap.add_argument("--out", default="profiles")
    ap.add_argument("--tag", default="gcn_rmat21")
    a = ap.parse_args()
    os.makedirs(a.out, exist_ok=True)

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
    for stage, (pats, src) in STAGES.items():
        parts = []
        for pat, per in pats[a.dtype]:
            keys = [k for k in set(fe) | set(wr) if k.startswith(pat)]
            if len(keys) != 1:
                break
            parts.append((keys[0], per))
        if len(parts) != len(pats[a.dtype]):
            continue
        entry = {"kernels": [], "source": src, "src_sha": src_sha(src), "bytes_per_launch": 0.0,
                 "trace_us_per_launch": 0.0, "calibration": {"fetch": cf, "write": cw}}
        for k, per in parts:
            f_ = sum(fe[k]) / len(fe[k])
            w_ = sum(wr[k]) / len(wr[k])
            n_avg = st.get(k, (0, 0.0, 0.0))[1]
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
