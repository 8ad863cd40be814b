"""Helpers for the measurements: source hashes and rocprofv3 output summaries.

``rocprofv3 --kernel-trace --stats --output-format csv`` writes a
``*_kernel_stats.csv``; ``rocprofv3 --pmc <counter> --output-format csv``
writes a ``*_counter_collection.csv`` with one row per (dispatch, counter).
FETCH_SIZE and WRITE_SIZE are reported in KiB per dispatch. Each is scaled by
the factor that makes a plain device-to-device copy of known size read and
write exactly its size, measured in the same counter run.

Command line (turns two counter runs into the traffic record bench.py reads):
  python -m paper_2608_21343_amd.profiling traffic FETCH_DIR WRITE_DIR KERNEL OUT.json [FIRST]
FIRST limits the mean to the kernel's first FIRST dispatches (in dispatch
order): with ``bench.py --steps 1 --warmup 0`` those are the timed step's
calls, before the bench's context measurements launch the kernel again.
"""

from __future__ import annotations

import csv
import glob
import hashlib
import json
import os
import sys
from typing import Dict, List, Optional

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# Sources that define the short-call greedy kernel (the streaming workload's
# dominant kernel); a traffic record is valid only for this exact text.
CHUNK_KERNEL_SOURCES = [
    "paper_2608_21343_amd/csrc/greedy_seg.hpp",
    "paper_2608_21343_amd/csrc/greedy_seg_17_24.hip",
    "paper_2608_21343_amd/csrc/device.hpp",
]

COPY_PROBE_BYTES = 256 << 20


def source_hash(paths: List[str] = CHUNK_KERNEL_SOURCES) -> str:
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def _find(d: str, suffix: str) -> str:
    hits = sorted(glob.glob(os.path.join(d, "**", "*" + suffix), recursive=True))
    if not hits:
        raise FileNotFoundError(f"no *{suffix} under {d}")
    return hits[-1]


def kernel_stats(d: str) -> List[Dict[str, object]]:
    """Rows of the kernel statistics csv under d, slowest total first."""
    with open(_find(d, "kernel_stats.csv")) as fh:
        rows = list(csv.DictReader(fh))
    out = []
    for r in rows:
        out.append({"name": r["Name"], "calls": int(r["Calls"]),
                    "total_ns": float(r["TotalDurationNs"]), "avg_ns": float(r["AverageNs"]),
                    "min_ns": float(r["MinNs"]), "max_ns": float(r["MaxNs"])})
    out.sort(key=lambda r: -r["total_ns"])
    return out


def counter_per_dispatch(d: str, counter: str) -> Dict[str, List[float]]:
    """Counter value of every dispatch under d, grouped by kernel name, in
    dispatch order."""
    with open(_find(d, "counter_collection.csv")) as fh:
        rows = list(csv.DictReader(fh))
    rows = [r for r in rows if r.get("Counter_Name") == counter]
    rows.sort(key=lambda r: int(r["Dispatch_Id"]))
    by: Dict[str, List[float]] = {}
    for r in rows:
        by.setdefault(r["Kernel_Name"], []).append(float(r["Counter_Value"]))
    return by


def _mean_for(by: Dict[str, List[float]], key: str, first: Optional[int] = None) -> float:
    names = [k for k in by if key in k]
    if len(names) != 1:
        raise KeyError(f"{len(names)} kernels match {key!r}")
    vals = by[names[0]][:first] if first else by[names[0]]
    return sum(vals) / len(vals)


def _copy_value(by: Dict[str, List[float]]) -> float:
    """The copy probe: the dispatch of a copy kernel with the largest count."""
    vals = [v for k, vs in by.items() if "copy" in k.lower() for v in vs]
    if not vals:
        raise KeyError("no copy kernel dispatch found (run bench.py with --copy-probe)")
    return max(vals)


def traffic_record(fetch_dir: str, write_dir: str, kernel: str,
                   first: Optional[int] = None) -> Dict[str, object]:
    f = counter_per_dispatch(fetch_dir, "FETCH_SIZE")
    w = counter_per_dispatch(write_dir, "WRITE_SIZE")
    kib = COPY_PROBE_BYTES / 1024.0
    f_scale = kib / _copy_value(f)
    w_scale = kib / _copy_value(w)
    fetch = _mean_for(f, kernel, first)
    write = _mean_for(w, kernel, first)
    return {
        "kernel": kernel,
        "dispatches": first or "all",
        "kernel_hash": source_hash(),
        "fetch_kib_per_dispatch": fetch,
        "write_kib_per_dispatch": write,
        "copy_fetch_scale": f_scale,
        "copy_write_scale": w_scale,
        "hbm_bytes_per_launch": (fetch * f_scale + write * w_scale) * 1024.0,
    }


def load_traffic(path: str) -> Optional[float]:
    """HBM bytes per launch from a traffic record, if it matches the current sources."""
    try:
        with open(path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    if rec.get("kernel_hash") != source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


def main(argv: List[str]) -> int:
    if len(argv) in (5, 6) and argv[0] == "traffic":
        rec = traffic_record(argv[1], argv[2], argv[3], int(argv[5]) if len(argv) == 6 else None)
        with open(argv[4], "w") as fh:
            json.dump(rec, fh, indent=1)
        print(json.dumps(rec))
        return 0
    if len(argv) == 2 and argv[0] == "stats":
        for r in kernel_stats(argv[1]):
            print(f"{r['calls']:6d} calls  avg {r['avg_ns'] / 1e3:10.2f} us  "
                  f"total {r['total_ns'] / 1e3:10.1f} us  {r['name'][:110]}")
        return 0
    print(__doc__)
    return 2


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
