"""Summaries of rocprofv3 output for the library's kernels.

    python -m paper_2508_09001_amd.profiling stats <dir> [--last N --kernel S]
        per-kernel dispatch count and duration (avg/min/max/total, microseconds)
        from a `rocprofv3 --kernel-trace --stats` output directory (CSV or the
        SQLite database rocprofv3 writes by default); with --last, also the
        average duration of the last N dispatches (by start time) of the kernels
        whose name contains S (bench.py ends with a graph of launches of its
        dominant kernel alone).

    python -m paper_2508_09001_amd.profiling traffic --kernel attend_kernel \\
        --fetch <dir> --write <dir> --calib-fetch <dir> --calib-write <dir> \\
        --calib-bytes N --sources f1 f2 ... --out <file.json>
        HBM bytes per dispatch of one kernel from two `rocprofv3 --pmc` runs
        (FETCH_SIZE, then WRITE_SIZE, KiB per dispatch), each scaled by what the
        same counter reads for a plain device copy of N bytes (N read, N
        written).  The JSON records the SHA-256 of the kernel's sources so that
        a reader can tell whether the counters still describe the built kernel.

Nothing here touches the GPU; it reads files only.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
import sqlite3
import sys
from collections import defaultdict


def sources_sha256(paths) -> str:
    h = hashlib.sha256()
    for p in paths:
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def _short(name: str) -> str:
    """Kernel name without return type, namespaces and parameter list."""
    if name.startswith("void "):
        name = name[5:]
    name = name.replace("retro::(anonymous namespace)::", "").replace("retro::", "")
    depth = 0
    for i, ch in enumerate(name):
        if ch == "<":
            depth += 1
        elif ch == ">":
            depth -= 1
        elif ch == "(" and depth == 0:
            return name[:i]
    return name


def kernel_durations(out_dir: str) -> dict:
    """kernel name -> list of durations (ns) of every dispatch."""
    res = defaultdict(list)
    trace = glob.glob(os.path.join(out_dir, "**", "*kernel_trace.csv"), recursive=True)
    if trace:
        for path in trace:
            with open(path, newline="") as f:
                for row in csv.DictReader(f):
                    res[row["Kernel_Name"]].append(
                        int(row["End_Timestamp"]) - int(row["Start_Timestamp"]))
        return res
    dbs = glob.glob(os.path.join(out_dir, "**", "*.db"), recursive=True)
    if not dbs:
        raise FileNotFoundError(f"no kernel trace under {out_dir}")
    for db in dbs:
        con = sqlite3.connect(db)
        for name, start, end in con.execute("select name, start, end from kernels"):
            res[name].append(int(end) - int(start))
        con.close()
    return res


def stats_table(out_dir: str) -> str:
    durs = kernel_durations(out_dir)
    rows = sorted(durs.items(), key=lambda kv: -sum(kv[1]))
    lines = ["| kernel | dispatches | avg us | min us | max us | total us |",
             "|---|---|---|---|---|---|"]
    for name, d in rows:
        lines.append(f"| {_short(name)} | {len(d)} | {sum(d) / len(d) / 1e3:.2f} | "
                     f"{min(d) / 1e3:.2f} | {max(d) / 1e3:.2f} | {sum(d) / 1e3:.1f} |")
    return "\n".join(lines)


def last_dispatches_avg(out_dir: str, kernel_substr: str, n: int) -> tuple:
    """(count, average duration in us) of the last n dispatches, by start time,
    of the kernels whose name contains kernel_substr (CSV kernel trace)."""
    spans = []
    for path in glob.glob(os.path.join(out_dir, "**", "*kernel_trace.csv"), recursive=True):
        with open(path, newline="") as f:
            for row in csv.DictReader(f):
                if kernel_substr in row["Kernel_Name"]:
                    spans.append((int(row["Start_Timestamp"]), int(row["End_Timestamp"])))
    spans.sort()
    last = spans[-n:] if n > 0 else []
    if not last:
        return 0, float("nan")
    return len(last), sum(e - s for s, e in last) / len(last) / 1e3


def counter_per_dispatch(out_dir: str, counter: str, kernel_substr: str) -> list:
    """Values of `counter` (summed over its instances) for every dispatch whose
    kernel name contains `kernel_substr`."""
    per = defaultdict(float)
    files = glob.glob(os.path.join(out_dir, "**", "*counter_collection.csv"), recursive=True)
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {out_dir}")
    for path in files:
        with open(path, newline="") as f:
            for row in csv.DictReader(f):
                if row.get("Counter_Name") != counter:
                    continue
                if kernel_substr not in row.get("Kernel_Name", ""):
                    continue
                key = (path, row.get("Dispatch_Id") or row.get("Correlation_Id"))
                per[key] += float(row["Counter_Value"])
    return list(per.values())


def traffic(args) -> dict:
    fetch = counter_per_dispatch(args.fetch, "FETCH_SIZE", args.kernel)
    write = counter_per_dispatch(args.write, "WRITE_SIZE", args.kernel)
    cf = counter_per_dispatch(args.calib_fetch, "FETCH_SIZE", args.calib_kernel)
    cw = counter_per_dispatch(args.calib_write, "WRITE_SIZE", args.calib_kernel)
    if not (fetch and write and cf and cw):
        raise SystemExit("missing dispatches: "
                         f"fetch {len(fetch)} write {len(write)} calib {len(cf)}/{len(cw)}")
    kib = 1024.0
    f_fac = args.calib_bytes / (max(cf) * kib)
    w_fac = args.calib_bytes / (max(cw) * kib)
    fetch_b = sum(fetch) / len(fetch) * kib * f_fac
    write_b = sum(write) / len(write) * kib * w_fac
    return {
        "kernel": args.kernel,
        "dispatches": {"fetch": len(fetch), "write": len(write)},
        "fetch_kib_per_dispatch_raw": round(sum(fetch) / len(fetch), 1),
        "write_kib_per_dispatch_raw": round(sum(write) / len(write), 1),
        "calib_copy_bytes": args.calib_bytes,
        "calib_fetch_kib_raw": max(cf),
        "calib_write_kib_raw": max(cw),
        "fetch_scale": round(f_fac, 4),
        "write_scale": round(w_fac, 4),
        "hbm_fetch_bytes_per_launch": int(fetch_b),
        "hbm_write_bytes_per_launch": int(write_b),
        "hbm_bytes_per_launch": int(fetch_b + write_b),
        "source_sha256": sources_sha256(args.sources),
        "sources": [os.path.relpath(p) for p in args.sources],
    }


def main(argv=None):
    p = argparse.ArgumentParser(description="rocprofv3 summaries")
    sub = p.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("dir")
    s.add_argument("--last", type=int, default=0)
    s.add_argument("--kernel", default="")
    t = sub.add_parser("traffic")
    t.add_argument("--kernel", required=True)
    t.add_argument("--fetch", required=True)
    t.add_argument("--write", required=True)
    t.add_argument("--calib-fetch", required=True)
    t.add_argument("--calib-write", required=True)
    t.add_argument("--calib-kernel", default="elementwise")
    t.add_argument("--calib-bytes", type=int, required=True)
    t.add_argument("--sources", nargs="+", required=True)
    t.add_argument("--out")
    a = p.parse_args(argv)
    if a.cmd == "stats":
        print(stats_table(a.dir))
        if a.last > 0:
            n, avg = last_dispatches_avg(a.dir, a.kernel, a.last)
            print(f"\nlast {n} dispatches of {a.kernel}: {avg:.2f} us average")
        return
    res = traffic(a)
    text = json.dumps(res, indent=1)
    if a.out:
        with open(a.out, "w") as f:
            f.write(text + "\n")
    print(text)


if __name__ == "__main__":
    sys.exit(main())
