"""Summaries of rocprofv3 output for the benchmark's kernels.

    python -m paper_2608_11231_amd.rocprof_summary trace  <kernel_trace.csv> <out.txt> <command...>
    python -m paper_2608_11231_amd.rocprof_summary traffic <fetch_counter_collection.csv> \
        <write_counter_collection.csv> <copy_bytes> <out.txt> <command...>

``traffic`` calibrates FETCH_SIZE / WRITE_SIZE on the plain device copy that
``bench.py --copy-probe`` launches (copy_bytes read and written), scales every
kernel's per-dispatch counters by those factors and records the hash of the
kernel sources, so that a reader can tell whether the counters still describe
the current kernels (``kernel_source_hash``).
"""
from __future__ import annotations

import collections
import csv
import glob
import hashlib
import os
import sys

HERE = os.path.dirname(os.path.abspath(__file__))


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in sorted(glob.glob(os.path.join(HERE, "csrc", "*"))):
        with open(p, "rb") as f:
            h.update(os.path.basename(p).encode())
            h.update(f.read())
    return h.hexdigest()[:16]


def short_name(name: str) -> str:
    name = name.replace("void ", "")
    name = name.split("(")[0] if "(" in name else name
    return name.replace(" ", "")


def trace(trace_csv: str, out: str, command: str) -> None:
    """Per (kernel, grid) dispatch durations from a --kernel-trace CSV: count,
    median, mean, min, max.  The median separates a kernel's steady-state
    launches from a one-off launch of the same symbol and grid."""
    groups = collections.defaultdict(list)
    for r in csv.DictReader(open(trace_csv)):
        grid = int(r["Grid_Size_X"]) * int(r["Grid_Size_Y"]) * int(r["Grid_Size_Z"])
        dur = (int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) / 1e3
        groups[(short_name(r["Kernel_Name"]), grid)].append(dur)
    lines = ["# rocprofv3 kernel trace, per-dispatch durations (us)", f"command: {command}",
             f"kernel_source_hash: {kernel_source_hash()}", "",
             f"{'kernel':60s} {'grid':>9s} {'calls':>6s} {'median_us':>10s} {'mean_us':>10s} {'min_us':>10s} "
             f"{'max_us':>10s}"]
    for (name, grid), d in sorted(groups.items(), key=lambda kv: -sum(kv[1])):
        d = sorted(d)
        med = d[len(d) // 2]
        lines.append(f"{name[:60]:60s} {grid:9d} {len(d):6d} {med:10.2f} {sum(d) / len(d):10.2f} {d[0]:10.2f} "
                     f"{d[-1]:10.2f}")
    open(out, "w").write("\n".join(lines) + "\n")


def _per_dispatch(path: str):
    rows = list(csv.DictReader(open(path)))
    out = []
    for r in rows:
        out.append((int(r["Dispatch_Id"]), r["Kernel_Name"], int(r["Grid_Size"]), float(r["Counter_Value"])))
    return out


def traffic(fetch_csv: str, write_csv: str, copy_bytes: int, out: str, command: str) -> None:
    fetch = _per_dispatch(fetch_csv)
    write = _per_dispatch(write_csv)

    def copy_kib(rows):
        vals = [v for _, name, grid, v in rows if "copyBuffer" in name and v * 1024 > copy_bytes / 8]
        return max(vals) if vals else None

    f_copy, w_copy = copy_kib(fetch), copy_kib(write)
    half = copy_bytes / 2 / 1024  # the probe reads and writes copy_bytes/2 each
    f_scale = half / f_copy if f_copy else None
    w_scale = half / w_copy if w_copy else None
    groups = collections.defaultdict(lambda: [[], []])
    for i, rows in ((0, fetch), (1, write)):
        for _, name, grid, v in rows:
            if "copyBuffer" in name or "elementwise" in name:
                continue
            groups[(short_name(name), grid)][i].append(v)
    lines = ["# rocprofv3 --pmc FETCH_SIZE and --pmc WRITE_SIZE (separate runs), per dispatch",
             f"command: {command}", f"kernel_source_hash: {kernel_source_hash()}",
             f"copy_probe_bytes: {copy_bytes}",
             f"fetch_scale: {f_scale:.4f}" if f_scale else "fetch_scale: none",
             f"write_scale: {w_scale:.4f}" if w_scale else "write_scale: none", "",
             f"{'kernel':60s} {'grid':>9s} {'fetch_KiB':>12s} {'write_KiB':>12s} {'traffic_bytes':>15s}"]
    for (name, grid), (fv, wv) in sorted(groups.items()):
        # medians: a kernel's repeated launches, not a one-off launch of the same symbol
        fk = sorted(fv)[len(fv) // 2] if fv else 0.0
        wk = sorted(wv)[len(wv) // 2] if wv else 0.0
        tb = (fk * (f_scale or 0) + wk * (w_scale or 0)) * 1024
        lines.append(f"{name[:60]:60s} {grid:9d} {fk:12.1f} {wk:12.1f} {tb:15.0f}")
    open(out, "w").write("\n".join(lines) + "\n")


def read_traffic(path: str):
    """{(kernel_name, grid): traffic_bytes} from a traffic summary, or None when
    the summary is missing or was taken on different kernel sources."""
    if not os.path.exists(path):
        return None
    lines = open(path).read().splitlines()
    meta = dict(l.split(": ", 1) for l in lines if ": " in l and not l.startswith("#"))
    if meta.get("kernel_source_hash") != kernel_source_hash():
        return None
    table = {}
    start = next((i for i, l in enumerate(lines) if l.startswith("kernel ")), None)
    if start is None:
        return None
    for l in lines[start + 1:]:
        parts = l.split()
        if len(parts) >= 5:
            table[(parts[0], int(parts[-4]))] = float(parts[-1])
    return table


if __name__ == "__main__":
    mode = sys.argv[1]
    if mode == "trace":
        trace(sys.argv[2], sys.argv[3], " ".join(sys.argv[4:]))
    elif mode == "traffic":
        traffic(sys.argv[2], sys.argv[3], int(sys.argv[4]), sys.argv[5], " ".join(sys.argv[6:]))
    else:
        raise SystemExit(__doc__)
