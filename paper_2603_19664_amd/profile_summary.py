"""Condense rocprofv3 CSV output into the short text summaries kept under profiles/.

    python -m paper_2603_19664_amd.profile_summary stats <run_kernel_stats.csv> "<command>" > profiles/X.md
    python -m paper_2603_19664_amd.profile_summary trace <run_kernel_trace.csv> "<command>" > profiles/X.md
    python -m paper_2603_19664_amd.profile_summary pmc <dir with p*/run_counter_collection.csv> <kernel substring> "<command>"
    python -m paper_2603_19664_amd.profile_summary pmc_by_grid <dir>[,<dir>...] <kernel substring> "<command>"
    python -m paper_2603_19664_amd.profile_summary pmc_seq <dir>[,<dir>...] <kernel> <block> <label,...> "<command>" [<copy kernel> <copy bytes>]
    python -m paper_2603_19664_amd.profile_summary sweep_traffic <fetch dir> <write dir> <trace csv> <kernel> <block> <label,...> <copy kernel> <copy bytes> "<command>"
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


def _rows(directory):
    for p in sorted(glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)):
        yield from csv.DictReader(open(p))


def _wgs(r):
    grid = r.get("Grid_Size") or r.get("Grid_Size_X") or "0"
    wg = r.get("Workgroup_Size") or r.get("Workgroup_Size_X") or "1"
    return int(grid) // max(int(wg), 1)


def pmc_by_grid(directories, kernel: str, command: str) -> str:
    """Mean per dispatch of every counter of `kernel`, one row per grid size (the number
    of workgroups tells the workload shapes of one run apart)."""
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    for d in directories:
        for r in _rows(d):
            if kernel in r["Kernel_Name"]:
                agg[_wgs(r)][r["Counter_Name"]].append(float(r["Counter_Value"]))
    names = sorted({c for g in agg.values() for c in g})
    out = ["# rocprofv3 counters per grid", "", f"Kernel: `{kernel}`", "",
           "Command (repository root, one MI355X; one rocprofv3 run per counter group):", "", "```", command, "```", "",
           "| workgroups | dispatches | " + " | ".join(names) + " |", "|---" * (len(names) + 2) + "|"]
    for wgs in sorted(agg):
        g = agg[wgs]
        n = max(len(v) for v in g.values())
        out.append(f"| {wgs} | {n} | " + " | ".join(f"{sum(g[c]) / len(g[c]):.6g}" if g.get(c) else "-"
                                                     for c in names) + " |")
    return "\n".join(out) + "\n"


def pmc_seq(directories, kernel: str, block: int, labels, command: str, copy_kernel: str = "",
            copy_bytes: int = 0) -> str:
    """Counters of `kernel` in dispatch order, `block` consecutive dispatches per label (a sweep
    that launches the kernel `block` times per point, points in the order of `labels`).  With a
    calibration copy (copy_kernel, copy_bytes: the largest dispatch of that kernel in each run),
    FETCH_SIZE and WRITE_SIZE are also given in bytes per dispatch."""
    agg = collections.defaultdict(lambda: collections.defaultdict(list))
    scale = {}
    for d in directories:
        rows = sorted(_rows(d), key=lambda r: int(r["Dispatch_Id"]))
        seen = collections.defaultdict(int)
        for r in rows:
            c = r["Counter_Name"]
            # the calibration copy is the run's first dispatch of the copy kernel
            if copy_kernel and copy_kernel in r["Kernel_Name"] and c in ("FETCH_SIZE", "WRITE_SIZE") and c not in scale:
                scale[c] = float(r["Counter_Value"])
            if kernel in r["Kernel_Name"]:
                i = seen[c]
                seen[c] += 1
                if i // block < len(labels):
                    agg[labels[i // block]][c].append(float(r["Counter_Value"]))
    names = sorted({c for g in agg.values() for c in g})
    extra = [f"{c} bytes" for c in ("FETCH_SIZE", "WRITE_SIZE") if c in names and c in scale]
    out = ["# rocprofv3 counters per sweep point", "", f"Kernel: `{kernel}`, {block} dispatches per point, in order: "
           + ", ".join(labels), "", "Command (repository root, one MI355X; one rocprofv3 run per counter group):", "",
           "```", command, "```", ""]
    if extra:
        out += [f"FETCH_SIZE / WRITE_SIZE (KiB) scaled to bytes by a {copy_bytes}-byte copy in the same run "
                f"({', '.join(f'{c} {scale[c]:.0f} KiB' for c in scale)}).", ""]
    out += ["| point | dispatches | " + " | ".join(names + extra) + " |", "|---" * (len(names) + len(extra) + 2) + "|"]
    for lab in labels:
        g = agg.get(lab)
        if not g:
            continue
        n = max(len(v) for v in g.values())
        vals = [f"{sum(g[c]) / len(g[c]):.6g}" if g.get(c) else "-" for c in names]
        for c in ("FETCH_SIZE", "WRITE_SIZE"):
            if f"{c} bytes" in extra:
                vals.append(f"{sum(g[c]) / len(g[c]) * copy_bytes / scale[c]:.4g}")
        out.append(f"| {lab} | {n} | " + " | ".join(vals) + " |")
    return "\n".join(out) + "\n"


def sweep_traffic(fetch_dir: str, write_dir: str, trace_csv: str, kernel: str, block: int, labels, copy_kernel: str,
                  copy_bytes: int, command: str, peak_gbs: float = 8000.0) -> str:
    """Per sweep point (block consecutive dispatches of `kernel` per label): the kernel-trace
    duration, FETCH_SIZE + WRITE_SIZE in bytes (scaled by the run's first copy-kernel dispatch,
    a copy of copy_bytes), and the HBM rate they give against peak_gbs."""
    def seq(rows, pick):
        out = collections.defaultdict(list)
        for i, v in enumerate(pick(r) for r in rows):
            if i // block < len(labels):
                out[labels[i // block]].append(v)
        return out

    def counter(directory, name):
        rows = sorted((r for r in _rows(directory) if r["Counter_Name"] == name), key=lambda r: int(r["Dispatch_Id"]))
        cal = next(float(r["Counter_Value"]) for r in rows if copy_kernel in r["Kernel_Name"])
        mine = [r for r in rows if kernel in r["Kernel_Name"]]
        return seq(mine, lambda r: float(r["Counter_Value"]) * copy_bytes / cal)

    tr = sorted((r for r in csv.DictReader(open(trace_csv)) if kernel in r["Kernel_Name"]),
                key=lambda r: int(r["Start_Timestamp"]))
    dur = seq(tr, lambda r: (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3)
    fe, wr = counter(fetch_dir, "FETCH_SIZE"), counter(write_dir, "WRITE_SIZE")
    out = ["# HBM traffic and rate per sweep point", "", f"Kernel: `{kernel}`, {block} dispatches per point, in order: "
           + ", ".join(labels), "", "Commands (repository root, one MI355X; a kernel trace and one counter run per counter):",
           "", "```", command, "```", "",
           f"Counter bytes are FETCH_SIZE / WRITE_SIZE scaled by the first `{copy_kernel}` dispatch of the same run (a "
           f"{copy_bytes}-byte copy).  Rate = (fetch + write) / mean trace duration; peak {peak_gbs:.0f} GB/s.", "",
           "| point | mean duration (us) | fetch (MB) | write (MB) | rate (GB/s) | fraction of peak |",
           "|---|---|---|---|---|---|"]
    for lab in labels:
        if not dur.get(lab):
            continue
        d = sum(dur[lab]) / len(dur[lab])
        f = sum(fe[lab]) / len(fe[lab])
        w = sum(wr[lab]) / len(wr[lab])
        gbs = (f + w) / (d * 1e-6) / 1e9
        out.append(f"| {lab} | {d:.1f} | {f / 1e6:.2f} | {w / 1e6:.3f} | {gbs:.0f} | {gbs / peak_gbs:.3f} |")
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
                    v.append((int(r["Dispatch_Id"]), float(r["Counter_Value"])))
        if not v:
            raise SystemExit(f"no {counter} samples for {name} under {directory}")
        return [x for _, x in sorted(v)]
    fv = values(fetch_dir, "FETCH_SIZE", kernel)
    wv = values(write_dir, "WRITE_SIZE", kernel)
    f_k, nf, w_k, nw = sum(fv) / len(fv), len(fv), sum(wv) / len(wv), len(wv)
    # the calibration copy is the run's first dispatch of the copy kernel (made before anything else)
    f_c = values(fetch_dir, "FETCH_SIZE", copy_kernel)[0]
    w_c = values(write_dir, "WRITE_SIZE", copy_kernel)[0]
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
    elif mode == "pmc_by_grid":
        sys.stdout.write(pmc_by_grid(sys.argv[2].split(","), sys.argv[3], sys.argv[4]))
    elif mode == "pmc_seq":
        dirs, kernel, block, labels, command = sys.argv[2:7]
        copy_kernel, copy_bytes = (sys.argv[7], int(sys.argv[8])) if len(sys.argv) > 8 else ("", 0)
        sys.stdout.write(pmc_seq(dirs.split(","), kernel, int(block), labels.split(","), command, copy_kernel,
                                 copy_bytes))
    elif mode == "sweep_traffic":
        fetch_dir, write_dir, trace_csv, kernel, block, labels, copy_kernel, copy_bytes, command = sys.argv[2:11]
        sys.stdout.write(sweep_traffic(fetch_dir, write_dir, trace_csv, kernel, int(block), labels.split(","),
                                       copy_kernel, int(copy_bytes), command))
    elif mode == "traffic":
        import json
        fetch_dir, write_dir, kernel, copy_kernel, copy_bytes, workload, command = sys.argv[2:9]
        sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
        from bench import source_hash
        print(json.dumps(traffic(fetch_dir, write_dir, kernel, copy_kernel, int(copy_bytes), workload, source_hash(),
                                 command), indent=1))
    else:
        raise SystemExit(__doc__)
