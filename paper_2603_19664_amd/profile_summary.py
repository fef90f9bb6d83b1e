"""Condense rocprofv3 CSV output into the short text summaries kept under profiles/.

    python -m paper_2603_19664_amd.profile_summary stats <run_kernel_stats.csv> "<command>" > profiles/X.md
    python -m paper_2603_19664_amd.profile_summary trace <run_kernel_trace.csv> "<command>" > profiles/X.md
    python -m paper_2603_19664_amd.profile_summary pmc <dir with p*/run_counter_collection.csv> <kernel substring> "<command>"
    python -m paper_2603_19664_amd.profile_summary traffic <fetch dir> <write dir> <kernel> <copy kernel> <copy bytes> <workload> "<command>"
"""
from __future__ import annotations

import collections
import csv
import glob
import os
import sys


def stats(path: str, command: str, top: int = 12) -> str:
    rows = list(csv.DictReader(open(path)))
    out = ["# rocprofv3 kernel statistics", "", "Command (repository root, one MI355X):", "", "```", command, "```", "",
           "| kernel | calls | average (us) | min (us) | max (us) | % of GPU time |", "|---|---|---|---|---|---|"]
    for r in rows[:top]:
        name = r["Name"].split("(")[0][:80]
        out.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.2f} | {float(r['MinNs']) / 1e3:.2f} | "
                   f"{float(r['MaxNs']) / 1e3:.2f} | {float(r['Percentage']):.1f} |")
    return "\n".join(out) + "\n"


def trace(path: str, command: str, top: int = 12) -> str:
    """Per (kernel, grid size) launch durations from a --kernel-trace CSV: kernels
    launched at several shapes get a row per shape."""
    groups = collections.defaultdict(list)
    for r in csv.DictReader(open(path)):
        grid = r.get("Grid_Size_X") or r.get("Grid_Size") or "?"
        wg = r.get("Workgroup_Size_X") or r.get("Workgroup_Size") or "1"
        groups[(r["Kernel_Name"].split("(")[0][:80], int(grid) // max(int(wg), 1))].append(
            (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    out = ["# rocprofv3 kernel trace, per kernel and grid", "", "Command (repository root, one MI355X):", "", "```",
           command, "```", "", "| kernel | workgroups | launches | average (us) | min (us) | max (us) |",
           "|---|---|---|---|---|---|"]
    for (name, wgs), v in sorted(groups.items(), key=lambda x: -sum(x[1]))[:top]:
        out.append(f"| `{name}` | {wgs} | {len(v)} | {sum(v) / len(v):.1f} | {min(v):.1f} | {max(v):.1f} |")
    return "\n".join(out) + "\n"


def pmc(directory: str, kernel: str, command: str) -> str:
    agg = collections.defaultdict(list)
    for p in sorted(glob.glob(os.path.join(directory, "p*", "run_counter_collection.csv"))):
        for r in csv.DictReader(open(p)):
            if kernel in r["Kernel_Name"]:
                agg[r["Counter_Name"]].append(float(r["Counter_Value"]))
    out = ["# rocprofv3 counters", "", f"Kernel: `{kernel}`", "", "Command (repository root, one MI355X; one rocprofv3 run per counter group):",
           "", "```", command, "```", "", "| counter | dispatches | mean per dispatch |", "|---|---|---|"]
    for k in sorted(agg):
        v = agg[k]
        out.append(f"| {k} | {len(v)} | {sum(v) / len(v):.6g} |")
    return "\n".join(out) + "\n"


def traffic(fetch_dir: str, write_dir: str, kernel: str, copy_kernel: str, copy_bytes: int, workload: str,
            source_hash: str, command: str) -> dict:
    """Per-launch HBM bytes of `kernel` from a FETCH_SIZE run and a WRITE_SIZE run, each scaled by
    what the same counter reads for a plain copy of copy_bytes bytes in the same run."""
    def values(directory, counter, name):
        v = []
        for p in glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(p)):
                if name in r["Kernel_Name"] and r["Counter_Name"] == counter:
                    v.append(float(r["Counter_Value"]))
        if not v:
            raise SystemExit(f"no {counter} samples for {name} under {directory}")
        return v
    fv = values(fetch_dir, "FETCH_SIZE", kernel)
    wv = values(write_dir, "WRITE_SIZE", kernel)
    f_k, nf, w_k, nw = sum(fv) / len(fv), len(fv), sum(wv) / len(wv), len(wv)
    # the calibration copy is the largest dispatch of the copy kernel in the run
    f_c = max(values(fetch_dir, "FETCH_SIZE", copy_kernel))
    w_c = max(values(write_dir, "WRITE_SIZE", copy_kernel))
    ff = copy_bytes / (f_c * 1024.0)
    fw = copy_bytes / (w_c * 1024.0)
    fetch = f_k * 1024.0 * ff
    write = w_k * 1024.0 * fw
    return {"workload": workload, "kernel": kernel, "source_hash": source_hash, "bytes_per_launch": fetch + write,
            "fetch_bytes": fetch, "write_bytes": write, "fetch_kib_raw": f_k, "write_kib_raw": w_k,
            "copy_bytes": copy_bytes, "copy_fetch_kib": f_c, "copy_write_kib": w_c, "fetch_scale": ff, "write_scale": fw,
            "dispatches": [nf, nw], "command": command}


if __name__ == "__main__":
    mode = sys.argv[1]
    if mode == "stats":
        sys.stdout.write(stats(sys.argv[2], sys.argv[3]))
    elif mode == "trace":
        sys.stdout.write(trace(sys.argv[2], sys.argv[3]))
    elif mode == "pmc":
        sys.stdout.write(pmc(sys.argv[2], sys.argv[3], sys.argv[4]))
    elif mode == "traffic":
        import json
        fetch_dir, write_dir, kernel, copy_kernel, copy_bytes, workload, command = sys.argv[2:9]
        sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
        from bench import source_hash
        print(json.dumps(traffic(fetch_dir, write_dir, kernel, copy_kernel, int(copy_bytes), workload, source_hash(),
                                 command), indent=1))
    else:
        raise SystemExit(__doc__)
