"""Summaries of rocprofv3 output for profiles/.

kernel-trace (``rocprofv3 --kernel-trace --stats``): per-kernel dispatch
count and mean / min / max duration from the ``*_kernel_stats.csv`` file.

counters (``rocprofv3 --pmc FETCH_SIZE`` and ``--pmc WRITE_SIZE``): mean KiB
per dispatch of a kernel, read from ``*_counter_collection.csv``.  HBM bytes
of a kernel = its counter reading x (known bytes of a plain copy / the copy
kernel's reading of the same counter).

  python -m paper_2506_01374_amd.profiling stats DIR [--kernel NAME]
  python -m paper_2506_01374_amd.profiling counter DIR COUNTER KERNEL_SUBSTRING
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


def counter_per_dispatch(dirpath: str, counter: str, kernel_sub: str) -> Dict[str, float]:
    """Mean value of `counter` per dispatch of kernels whose name contains kernel_sub."""
    vals: Dict[int, float] = {}
    name = None
    for path in _find(dirpath, "counter_collection.csv"):
        with open(path) as f:
            for r in csv.DictReader(f):
                kn = r.get("Kernel_Name", "")
                if kernel_sub not in kn or r.get("Counter_Name") != counter:
                    continue
                name = kn
                d = int(r.get("Dispatch_Id", len(vals)))
                vals[d] = vals.get(d, 0.0) + float(r.get("Counter_Value", 0.0))
    if not vals:
        return {"kernel": None, "dispatches": 0, "mean": float("nan")}
    v = list(vals.values())
    return {"kernel": name, "dispatches": len(v), "mean": sum(v) / len(v), "min": min(v), "max": max(v)}


def main(argv=None):
    argv = argv or sys.argv[1:]
    if argv[:1] == ["stats"]:
        for r in kernel_stats(argv[1]):
            print(f"{r['name'][:60]:60s} calls={r['calls']:6d} avg={r['avg_ns'] / 1e3:9.3f} us "
                  f"min={r['min_ns'] / 1e3:9.3f} max={r['max_ns'] / 1e3:9.3f} ({r['pct']:.1f}%)")
    elif argv[:1] == ["counter"]:
        print(counter_per_dispatch(argv[1], argv[2], argv[3]))
    else:
        print(__doc__)


if __name__ == "__main__":
    main()
