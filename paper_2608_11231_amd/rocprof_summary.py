"""Summaries of rocprofv3 output for the benchmark's kernels.

    python -m paper_2608_11231_amd.rocprof_summary trace  <kernel_trace.csv> <out.txt> <command...>
    python -m paper_2608_11231_amd.rocprof_summary traffic <fetch_counter_collection.csv> \
        <write_counter_collection.csv> <copy_bytes> <out.txt> <command...>

    python -m paper_2608_11231_amd.rocprof_summary counters <out.txt> <counter_collection.csv>... -- <command...>

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


def _counter_rows(path: str):
    """(dispatch, kernel, grid, counter, value, duration_ns, vgpr, agpr, lds) per row
    of a rocprofv3 --pmc CSV (one row per dispatch and counter)."""
    out = []
    for r in csv.DictReader(open(path)):
        dur = None
        if r.get("Start_Timestamp") and r.get("End_Timestamp"):
            dur = int(r["End_Timestamp"]) - int(r["Start_Timestamp"])
        out.append((int(r["Dispatch_Id"]), short_name(r["Kernel_Name"]), int(r["Grid_Size"]), r["Counter_Name"],
                    float(r["Counter_Value"]), dur, r.get("VGPR_Count", ""), r.get("Accum_VGPR_Count", ""),
                    r.get("LDS_Block_Size", "")))
    return out


# CDNA4 (MI355X): 8 XCDs, 256 compute units of 4 SIMDs
N_XCD, N_CU, N_SIMD = 8, 256, 1024


def counters(out: str, paths, command: str) -> None:
    """Per (kernel, grid): the median over its dispatches of every SQ/GRBM counter
    in the given --pmc runs, and derived shares of the dispatch's cycles.
    GRBM_GUI_ACTIVE is summed over the 8 XCDs, so the dispatch's cycles are
    GRBM_GUI_ACTIVE / 8 (``clock_GHz`` checks that against the dispatch time).
    A wave64 VALU instruction holds its SIMD for 4 cycles, and
    SQ_ACTIVE_INST_VALU counts about one unit per instruction, i.e. quad-cycles:
      mfma_busy    = SQ_VALU_MFMA_BUSY_CYCLES / (cycles * 1024 SIMDs)
      valu_busy    = 4 * SQ_ACTIVE_INST_VALU / (cycles * 1024 SIMDs)
      lds_busy     = SQ_LDS_IDX_ACTIVE / (cycles * 256 CUs)
      lds_conflict = SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE (share of the LDS's
                     active cycles lost to bank conflicts)
    and per-wave instruction counts (SQ_INSTS_* / SQ_WAVES)."""
    groups = collections.defaultdict(lambda: collections.defaultdict(list))
    meta = {}
    for p in paths:
        for _, name, grid, cname, val, dur, vg, ag, lds in _counter_rows(p):
            groups[(name, grid)][cname].append(val)
            if dur is not None:
                groups[(name, grid)]["duration_us"].append(dur / 1e3)
            meta[(name, grid)] = (vg, ag, lds)

    def med(v):
        v = sorted(v)
        return v[len(v) // 2] if v else None

    lines = ["# rocprofv3 --pmc SQ/GRBM counters, per dispatch (median over a kernel's dispatches)",
             f"command: {command}", f"kernel_source_hash: {kernel_source_hash()}",
             "derived: cycles = GRBM_GUI_ACTIVE / 8 XCDs; mfma_busy = SQ_VALU_MFMA_BUSY_CYCLES / "
             "(cycles * 1024); valu_busy = 4 * SQ_ACTIVE_INST_VALU / (cycles * 1024); lds_busy = "
             "SQ_LDS_IDX_ACTIVE / (cycles * 256); lds_conflict = SQ_LDS_BANK_CONFLICT / SQ_LDS_IDX_ACTIVE; "
             "per_wave = SQ_INSTS_* / SQ_WAVES", ""]
    for (name, grid), cs in sorted(groups.items()):
        if not name.startswith("lkv::"):
            continue
        m = {k: med(v) for k, v in cs.items()}
        vg, ag, lds = meta[(name, grid)]
        lines.append(f"kernel {name}  grid {grid}  vgpr {vg}  agpr {ag}  lds {lds}  dispatches "
                     f"{max(len(v) for v in cs.values())}")
        for k in sorted(m):
            lines.append(f"  {k:34s} {m[k]:.6g}")
        der = []
        gui = m.get("GRBM_GUI_ACTIVE")
        if gui:
            cyc = gui / N_XCD
            if m.get("duration_us"):
                der.append(f"clock_GHz {cyc / (m['duration_us'] * 1e3):.2f}")
            if m.get("SQ_VALU_MFMA_BUSY_CYCLES") is not None:
                der.append(f"mfma_busy {m['SQ_VALU_MFMA_BUSY_CYCLES'] / (cyc * N_SIMD):.3f}")
            if m.get("SQ_ACTIVE_INST_VALU") is not None:
                der.append(f"valu_busy {4 * m['SQ_ACTIVE_INST_VALU'] / (cyc * N_SIMD):.3f}")
            if m.get("SQ_LDS_IDX_ACTIVE") is not None:
                der.append(f"lds_busy {m['SQ_LDS_IDX_ACTIVE'] / (cyc * N_CU):.3f}")
        if m.get("SQ_LDS_BANK_CONFLICT") is not None and m.get("SQ_LDS_IDX_ACTIVE"):
            der.append(f"lds_conflict {m['SQ_LDS_BANK_CONFLICT'] / m['SQ_LDS_IDX_ACTIVE']:.3f}")
        waves = m.get("SQ_WAVES")
        if waves:
            for k in sorted(m):
                if k.startswith("SQ_INSTS_"):
                    der.append(f"{k[len('SQ_INSTS_'):].lower()}_per_wave {m[k] / waves:.1f}")
        if der:
            lines.append("  derived: " + "; ".join(der))
        lines.append("")
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
    elif mode == "counters":
        sep = sys.argv.index("--")
        counters(sys.argv[2], sys.argv[3:sep], " ".join(sys.argv[sep + 1:]))
    else:
        raise SystemExit(__doc__)
