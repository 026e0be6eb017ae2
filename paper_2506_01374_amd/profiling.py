"""Summaries of rocprofv3 output for profiles/.

kernel-trace (``rocprofv3 --kernel-trace --stats``): per-kernel dispatch
count and mean / min / max duration from the ``*_kernel_stats.csv`` file.

counters (``rocprofv3 --pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE``): mean KiB
per dispatch of a kernel, read from ``*_counter_collection.csv``.  HBM bytes
of a kernel = its counter reading x (known bytes of a plain copy / the copy
kernel's reading of the same counter).

  python -m paper_2506_01374_amd.profiling stats DIR [--kernel NAME]
  python -m paper_2506_01374_amd.profiling dispatches DIR
  python -m paper_2506_01374_amd.profiling counter DIR COUNTER KERNEL_SUBSTRING [GRID_THREADS]
  python -m paper_2506_01374_amd.profiling traffic --workload NAME --schedule KEY \
      --kernel SUBSTRING --source FILE --fetch DIR --write DIR --cal-fetch DIR \
      --cal-write DIR --copy-bytes N [--copy-kernel SUBSTRING] [--command CMD ...] \
      --out profiles/traffic.json

``traffic`` converts the two counter runs of a kernel and the two runs of
a plain copy of N bytes into HBM bytes per launch and records them, keyed
by workload, with the schedule and the sha1 of the kernel source they were
taken for (the benchmark reports them only while both still match).
"""
from __future__ import annotations

import csv
import glob
import os
import sys
from typing import Dict, List


def _find(dirpath: str, suffix: str) -> List[str]:
    return sorted(glob.glob(os.path.join(dirpath, "**", f"*{suffix}"), recursive=True))


def kernel_stats(dirpath: str) -> List[Dict[str, float]]:
    rows = []
    for path in _find(dirpath, "kernel_stats.csv"):
        with open(path) as f:
            for r in csv.DictReader(f):
                rows.append({"name": r.get("Name", ""), "calls": int(r.get("Calls", 0)),
                             "total_ns": float(r.get("TotalDurationNs", 0)),
                             "avg_ns": float(r.get("AverageNs", 0)),
                             "min_ns": float(r.get("MinNs", 0)), "max_ns": float(r.get("MaxNs", 0)),
                             "pct": float(r.get("Percentage", 0))})
    return rows


def dispatch_stats(dirpath: str) -> List[Dict[str, float]]:
    """Per (kernel name, code object, grid size in threads, workgroup size)
    duration statistics from the per-dispatch ``*_kernel_trace.csv``
    (launches of one kernel with different schedules share a name, not
    always a grid; each schedule is its own code object, with its own kernel
    id, for the duration of a run)."""
    groups: Dict[tuple, List[float]] = {}
    for path in _find(dirpath, "kernel_trace.csv"):
        with open(path) as f:
            for r in csv.DictReader(f):
                g = int(r.get("Grid_Size_X", 0)) * int(r.get("Grid_Size_Y", 1)) * int(r.get("Grid_Size_Z", 1))
                w = int(r.get("Workgroup_Size_X", 0)) * int(r.get("Workgroup_Size_Y", 1)) * \
                    int(r.get("Workgroup_Size_Z", 1))
                d = float(r["End_Timestamp"]) - float(r["Start_Timestamp"])
                groups.setdefault((r.get("Kernel_Name", ""), r.get("Kernel_Id", ""), g, w), []).append(d)
    out = []
    for (name, kid, g, w), ds in groups.items():
        out.append({"name": name, "kernel_id": kid, "grid_threads": g, "workgroup": w, "calls": len(ds),
                    "avg_ns": sum(ds) / len(ds), "min_ns": min(ds), "max_ns": max(ds)})
    return sorted(out, key=lambda r: -r["avg_ns"] * r["calls"])


def counter_per_dispatch(dirpath: str, counter: str, kernel_sub: str,
                         grid_threads: int = 0) -> Dict[str, float]:
    """Mean value of `counter` per dispatch of kernels whose name contains
    kernel_sub (and, if given, whose grid has grid_threads threads)."""
    vals: Dict[int, float] = {}
    name = None
    for path in _find(dirpath, "counter_collection.csv"):
        with open(path) as f:
            for r in csv.DictReader(f):
                kn = r.get("Kernel_Name", "")
                if kernel_sub not in kn or r.get("Counter_Name") != counter:
                    continue
                if grid_threads and int(r.get("Grid_Size", 0)) != grid_threads:
                    continue
                name = kn
                d = int(r.get("Dispatch_Id", len(vals)))
                vals[d] = vals.get(d, 0.0) + float(r.get("Counter_Value", 0.0))
    if not vals:
        return {"kernel": None, "dispatches": 0, "mean": float("nan")}
    v = list(vals.values())
    return {"kernel": name, "dispatches": len(v), "mean": sum(v) / len(v), "min": min(v), "max": max(v)}


def traffic_record(schedule: str, kernel_sub: str, source: str, fetch_dir: str, write_dir: str,
                   cal_fetch_dir: str, cal_write_dir: str, copy_bytes: int,
                   commands: List[str], copy_kernel: str = "copyBuffer",
                   grid_threads: int = 0) -> Dict[str, object]:
    import hashlib
    fk = counter_per_dispatch(fetch_dir, "FETCH_SIZE", kernel_sub, grid_threads)
    wk = counter_per_dispatch(write_dir, "WRITE_SIZE", kernel_sub, grid_threads)
    # the calibration runs also fill the source buffer; only the copy counts
    cf = counter_per_dispatch(cal_fetch_dir, "FETCH_SIZE", copy_kernel)
    cw = counter_per_dispatch(cal_write_dir, "WRITE_SIZE", copy_kernel)
    for what, r in (("kernel FETCH_SIZE", fk), ("kernel WRITE_SIZE", wk), ("copy FETCH_SIZE", cf),
                    ("copy WRITE_SIZE", cw)):
        if not r["dispatches"]:
            raise SystemExit(f"no dispatches found for {what}")
    fscale = copy_bytes / (cf["mean"] * 1024.0)
    wscale = copy_bytes / (cw["mean"] * 1024.0)
    fb = fk["mean"] * 1024.0 * fscale
    wb = wk["mean"] * 1024.0 * wscale
    return {"key": schedule, "kernel": fk["kernel"], "grid_threads": grid_threads or None,
            "kernel_source_sha1": hashlib.sha1(open(source, "rb").read()).hexdigest()[:16],
            "fetch_kib_per_dispatch": fk["mean"], "write_kib_per_dispatch": wk["mean"],
            "dispatches": [fk["dispatches"], wk["dispatches"]],
            "copy_reference_bytes": copy_bytes, "copy_kernel": cf["kernel"],
            "copy_fetch_kib": cf["mean"], "copy_write_kib": cw["mean"],
            "fetch_scale": fscale, "write_scale": wscale,
            "fetch_bytes_per_launch": fb, "write_bytes_per_launch": wb,
            "bytes_per_launch": fb + wb, "commands": commands}


def main(argv=None):
    argv = argv or sys.argv[1:]
    if argv[:1] == ["traffic"]:
        import argparse
        import json
        ap = argparse.ArgumentParser(prog="profiling traffic")
        for flag in ("--workload", "--schedule", "--kernel", "--source", "--fetch", "--write",
                     "--cal-fetch", "--cal-write", "--out"):
            ap.add_argument(flag, required=True)
        ap.add_argument("--copy-bytes", type=int, required=True)
        ap.add_argument("--copy-kernel", default="copyBuffer", help="name substring of the copy kernel")
        ap.add_argument("--grid-threads", type=int, default=0,
                        help="only dispatches of this many threads (kernels sharing a name)")
        ap.add_argument("--command", action="append", default=[])
        a = ap.parse_args(argv[1:])
        rec = traffic_record(a.schedule, a.kernel, a.source, a.fetch, a.write, a.cal_fetch,
                             a.cal_write, a.copy_bytes, a.command, a.copy_kernel, a.grid_threads)
        table = json.load(open(a.out)) if os.path.exists(a.out) else {}
        table[a.workload] = rec
        with open(a.out, "w") as f:
            json.dump(table, f, indent=2)
            f.write("\n")
        print(json.dumps({k: rec[k] for k in ("kernel", "fetch_kib_per_dispatch", "write_kib_per_dispatch",
                                              "fetch_scale", "bytes_per_launch")}))
        return
    if argv[:1] == ["stats"]:
        for r in kernel_stats(argv[1]):
            print(f"{r['name'][:60]:60s} calls={r['calls']:6d} avg={r['avg_ns'] / 1e3:9.3f} us "
                  f"min={r['min_ns'] / 1e3:9.3f} max={r['max_ns'] / 1e3:9.3f} ({r['pct']:.1f}%)")
    elif argv[:1] == ["dispatches"]:
        for r in dispatch_stats(argv[1]):
            print(f"{r['name'][:50]:50s} grid={r['grid_threads']:9d} wg={r['workgroup']:5d} calls={r['calls']:6d} "
                  f"avg={r['avg_ns'] / 1e3:9.3f} us min={r['min_ns'] / 1e3:9.3f} max={r['max_ns'] / 1e3:9.3f}")
    elif argv[:1] == ["counter"]:
        print(counter_per_dispatch(argv[1], argv[2], argv[3], int(argv[4]) if len(argv) > 4 else 0))
    else:
        print(__doc__)


if __name__ == "__main__":
    main()
