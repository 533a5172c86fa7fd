#!/usr/bin/env python3
"""rocprofv3 passes over bench.py and the summaries kept under profiles/.

  python profile_bench.py [--config 2] [--raw DIR]   (raw profiler output; default prof_raw/)

Three profiler runs of `bench.py --no-cpu` for one workload, each a child
process under its own time limit:
  1. --kernel-trace --stats: per-kernel call counts and durations;
  2. --pmc FETCH_SIZE: HBM bytes read per dispatch (KiB);
  3. --pmc WRITE_SIZE: HBM bytes written per dispatch (KiB).
bench.py also performs one device-to-device copy of 256 MiB (the last copy
before the first verify-step kernel); its counter readings give the scale
factors that turn each counter into bytes (the
counters need not count every byte once). The script writes
profiles/<entry point>_<workload>.md (command, kernel durations, calibrated
traffic per call) and updates profiles/counters.json, which bench.py reads
for the roofline's `traffic` (keyed by a hash of the kernel sources, so a
changed kernel reports null until it is profiled again).
Raw profiler output stays under --raw.
"""

from __future__ import annotations

import argparse
import collections
import csv
import glob
import json
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, HERE)

CAL_BYTES = 256 << 20  # bench.py's calibration copy
ENTRY_KERNELS = {  # kernel-name fragments launched by each entry point
    "verify_attention": ["attn_split_kernel", "attn_order_kernel"],
    "accept_and_diverge": ["accept_kernel", "accept_finish_kernel"],
    "rollback": ["rollback_kernel"],
    "accept_filter": ["accept_filter_kernel"],  # top-k / top-p thresholds (sampling variants only)
}
COPY_KERNEL = "copyBuffer"


def run(cmd, log, limit, kill_signal="TERM"):
    print("+", " ".join(cmd), flush=True)
    with open(log, "w") as f:
        rc = subprocess.run(["timeout", "-s", kill_signal, "-k", "10", str(limit)] + cmd, stdout=f,
                            stderr=subprocess.STDOUT, cwd="/tmp").returncode
    print(f"  rc={rc} log={log}", flush=True)
    return rc


def read_stats(d):
    files = glob.glob(os.path.join(d, "**", "*kernel_stats.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no kernel_stats.csv under {d}")
    return list(csv.DictReader(open(files[0])))


def read_counter(d, name):
    """Per-kernel-name list of counter values, and the calibration copy's value:
    the last copy dispatch before the first verify-step kernel."""
    files = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise SystemExit(f"no counter_collection.csv under {d}")
    rows = [r for r in csv.DictReader(open(files[0])) if r["Counter_Name"] == name]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    ours = [frag for frags in ENTRY_KERNELS.values() for frag in frags]
    first = next((i for i, r in enumerate(rows) if any(f in r["Kernel_Name"] for f in ours)), None)
    if first is None:
        raise SystemExit(f"no verify-step kernel in {files[0]}")
    cal = next((float(r["Counter_Value"]) for r in reversed(rows[:first]) if COPY_KERNEL in r["Kernel_Name"]), None)
    if cal is None:
        raise SystemExit(f"no calibration copy before the first verify-step kernel in {files[0]}")
    per = collections.defaultdict(list)
    for r in rows[first:]:
        per[r["Kernel_Name"]].append(float(r["Counter_Value"]))
    return per, cal


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--config", type=int, default=2)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--pmc-steps", type=int, default=10)
    ap.add_argument("--raw", default=os.path.join(HERE, "prof_raw"))
    ap.add_argument("--parse-only", action="store_true", help="summarise an earlier run's raw output")
    args = ap.parse_args()
    os.environ["TMPDIR"] = "/tmp"

    from bench import kernel_source_hash
    from workloads import CONFIGS

    workload = CONFIGS[args.config].name
    raw = os.path.join(os.path.abspath(args.raw), f"c{args.config}")
    os.makedirs(raw, exist_ok=True)
    bench = [sys.executable, os.path.join(HERE, "bench.py"), "--config", str(args.config), "--no-cpu"]
    cmd_trace = ["rocprofv3", "--kernel-trace", "--stats", "--output-format", "csv", "-d",
                 os.path.join(raw, "trace"), "-o", "run", "--"] + bench + ["--steps", str(args.steps),
                                                                         "--warmup", "10"]
    if not args.parse_only and run(cmd_trace, os.path.join(raw, "trace.log"), 600) != 0:
        raise SystemExit("kernel-trace pass failed")
    cmds_pmc = {}
    for ctr in ("FETCH_SIZE", "WRITE_SIZE"):
        cmds_pmc[ctr] = ["rocprofv3", "--pmc", ctr, "--output-format", "csv", "-d", os.path.join(raw, ctr), "-o",
                         "run", "--"] + bench + ["--steps", str(args.pmc_steps), "--warmup", "2"]
        if not args.parse_only and run(cmds_pmc[ctr], os.path.join(raw, ctr + ".log"), 300, kill_signal="KILL") != 0:
            raise SystemExit(f"{ctr} pass failed")

    stats = read_stats(os.path.join(raw, "trace"))
    fetch, cal_f = read_counter(os.path.join(raw, "FETCH_SIZE"), "FETCH_SIZE")
    write, cal_w = read_counter(os.path.join(raw, "WRITE_SIZE"), "WRITE_SIZE")

    def mean_kib(per, frag):
        """Mean over the dispatches of the kernel (full name, template
        arguments included) that contains frag and was dispatched most often:
        the verify step's instantiation, not a greedy or filtered variant."""
        names = [k for k in per if frag in k]
        if not names:
            return None, 0, None
        k = max(names, key=lambda n: len(per[n]))
        vals = per[k]
        return sum(vals) / len(vals), len(vals), k

    if cal_f <= 0 or cal_w <= 0:
        raise SystemExit("calibration copy reads zero")
    f_scale = CAL_BYTES / (cal_f * 1024)
    w_scale = CAL_BYTES / (cal_w * 1024)

    counters_path = os.path.join(HERE, "profiles", "counters.json")
    try:
        counters = json.load(open(counters_path))
    except (OSError, ValueError):
        counters = {}
    rel = lambda c: " ".join(os.path.relpath(x, HERE) if x.startswith(HERE) else x for x in c)  # noqa: E731
    for entry, frags in ENTRY_KERNELS.items():
        rows = [r for r in stats if any(fr in r["Name"] for fr in frags)]
        if not rows:
            continue
        total_f = total_w = 0.0
        lines = []
        for fr in frags:
            kf, nf, name = mean_kib(fetch, fr)
            kw, nw, _ = mean_kib(write, fr)
            if kf is None or kw is None:
                continue
            total_f += kf * 1024 * f_scale
            total_w += kw * 1024 * w_scale
            short = name.replace("(anonymous namespace)::", "").split("(")[0]
            lines.append(f"| {short[:90]} | {kf:.1f} | {kw:.1f} | {nf} |")
        per_call = int(round(total_f + total_w))
        counters.setdefault(entry, {})[workload] = {
            "source_hash": kernel_source_hash(entry), "bytes_per_call": per_call,
            "read_bytes": int(round(total_f)), "write_bytes": int(round(total_w)),
        }
        md = [f"# {entry} — {workload}", "",
              "Kernel trace (rocprofv3 --kernel-trace --stats), durations in microseconds:", "",
              "| kernel | calls | avg | min | max |", "|---|---|---|---|---|"]
        for r in rows:
            md.append(f"| {r['Name'][:90]} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | "
                      f"{float(r['MinNs']) / 1e3:.2f} | {float(r['MaxNs']) / 1e3:.2f} |")
        md += ["", "HBM counters per dispatch (KiB, raw):", "", "| kernel | FETCH_SIZE | WRITE_SIZE | dispatches |",
               "|---|---|---|---|"] + lines
        md += ["", f"Calibration: a {CAL_BYTES >> 20} MiB device copy reads FETCH_SIZE {cal_f:.0f} KiB and "
               f"WRITE_SIZE {cal_w:.0f} KiB; scale factors {f_scale:.4f} (read) and {w_scale:.4f} (write).",
               f"Calibrated HBM traffic per call: {total_f / 1e6:.2f} MB read + {total_w / 1e6:.2f} MB written "
               f"= {per_call / 1e6:.2f} MB.", f"Kernel source hash: {kernel_source_hash(entry)}.", "",
               f"Made by `python3 profile_bench.py --config {args.config} --raw <dir>` on the GPU, which runs "
               "(from /tmp, TMPDIR=/tmp):", "", "```", rel(cmd_trace)]
        md += [rel(c) for c in cmds_pmc.values()] + ["```", ""]
        with open(os.path.join(HERE, "profiles", f"{entry}_{workload}.md"), "w") as f:
            f.write("\n".join(md))
        print("\n".join(md), flush=True)
    with open(counters_path, "w") as f:
        json.dump(counters, f, indent=1, sort_keys=True)
        f.write("\n")


if __name__ == "__main__":
    main()
