"""Turn rocprofv3 CSV output into the short text summaries kept in profiles/.

``stats``: per-kernel call count and average / total duration from a
``--kernel-trace --stats`` run; with ``--trace`` the per-dispatch trace of the
same run is split by grid size, so that launches of one kernel on different
workloads are averaged apart. ``traffic``: HBM bytes per launch of one
kernel from two ``--pmc`` runs (FETCH_SIZE, then WRITE_SIZE, KiB per
dispatch), each scaled by what the same counter reads for a plain copy of a
known number of bytes; the summary records a hash of the kernel's source so
that a reader can tell whether the counters still describe the code.

The summaries are ``key = value`` text lines plus the command that produced
the profile.
"""
from __future__ import annotations

import argparse
import csv
import hashlib
import os
import statistics
from typing import Dict, List, Optional


def _rows(path: str) -> List[Dict[str, str]]:
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _col(row: Dict[str, str], *names: str) -> Optional[str]:
    for n in names:
        if n in row:
            return row[n]
    low = {k.lower(): v for k, v in row.items()}
    for n in names:
        if n.lower() in low:
            return low[n.lower()]
    return None


def source_hash(path: str) -> str:
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def kernel_stats(stats_csv: str) -> List[Dict[str, float]]:
    """Rows of a rocprofv3 *_kernel_stats.csv: name, calls, average and total ns."""
    out = []
    for r in _rows(stats_csv):
        name = _col(r, "Name", "KernelName", "Kernel_Name")
        calls = _col(r, "Calls")
        avg = _col(r, "AverageNs", "Average_ns", "Avg")
        tot = _col(r, "TotalDurationNs", "Total_ns", "TotalNs")
        if name is None or calls is None:
            continue
        out.append({"name": name, "calls": int(float(calls)),
                    "avg_ns": float(avg) if avg else float("nan"),
                    "total_ns": float(tot) if tot else float("nan")})
    return out


def counter_per_dispatch(counter_csv: str, kernel_substr: str, counter: str,
                         grid_size: Optional[int] = None) -> List[float]:
    """Counter values (summed over the per-dispatch rows) of dispatches whose
    kernel name contains ``kernel_substr`` (and, if given, of that grid size)."""
    per: Dict[str, float] = {}
    for r in _rows(counter_csv):
        name = _col(r, "Kernel_Name", "Kernel-Name", "KernelName") or ""
        cname = _col(r, "Counter_Name", "Counter-Name", "CounterName") or ""
        if kernel_substr not in name or cname != counter:
            continue
        if grid_size is not None and int(float(_col(r, "Grid_Size") or -1)) != grid_size:
            continue
        did = _col(r, "Dispatch_Id", "Dispatch-Id", "DispatchId") or str(len(per))
        per[did] = per.get(did, 0.0) + float(_col(r, "Counter_Value", "Counter-Value",
                                                   "CounterValue") or 0.0)
    return list(per.values())


def trace_by_grid(trace_csv: str) -> Dict[tuple, List[float]]:
    """Per (kernel, grid size): the durations (ns) of its dispatches."""
    out: Dict[tuple, List[float]] = {}
    for r in _rows(trace_csv):
        name = _col(r, "Kernel_Name") or ""
        gx = int(float(_col(r, "Grid_Size_X", "Grid_Size") or 0))
        gy = int(float(_col(r, "Grid_Size_Y") or 1))
        dur = float(_col(r, "End_Timestamp")) - float(_col(r, "Start_Timestamp"))
        out.setdefault((name, gx * gy), []).append(dur)
    return out


def cmd_stats(a) -> None:
    rows = kernel_stats(a.stats_csv)
    lines = [f"# rocprofv3 kernel stats: {a.title}", f"command = {a.command}", ""]
    for r in sorted(rows, key=lambda r: -r["total_ns"]):
        if a.kernel and not any(k in r["name"] for k in a.kernel):
            continue
        lines.append(f"kernel = {r['name']}")
        lines.append(f"  calls = {r['calls']}")
        lines.append(f"  average_us = {r['avg_ns'] / 1e3:.3f}")
        lines.append(f"  total_ms = {r['total_ns'] / 1e6:.3f}")
    if a.trace:
        lines.append("")
        lines.append("# per grid size (threads), from the kernel trace of the same run")
        for (name, grid), durs in sorted(trace_by_grid(a.trace).items()):
            if a.kernel and not any(k in name for k in a.kernel):
                continue
            lines.append(f"kernel = {name} grid_threads = {grid}")
            lines.append(f"  calls = {len(durs)}")
            lines.append(f"  average_us = {statistics.fmean(durs) / 1e3:.3f}")
            lines.append(f"  median_us = {statistics.median(durs) / 1e3:.3f}")
    _write(a.out, lines)


def cmd_traffic(a) -> None:
    fetch = counter_per_dispatch(a.fetch_csv, a.kernel, "FETCH_SIZE", a.grid_size)
    write = counter_per_dispatch(a.write_csv, a.kernel, "WRITE_SIZE", a.grid_size)
    cfetch = counter_per_dispatch(a.copy_fetch_csv, a.copy_kernel, "FETCH_SIZE")
    cwrite = counter_per_dispatch(a.copy_write_csv, a.copy_kernel, "WRITE_SIZE")
    if not (fetch and write and cfetch and cwrite):
        raise SystemExit("missing counter rows: "
                         f"{len(fetch)} {len(write)} {len(cfetch)} {len(cwrite)}")
    med = statistics.median
    # a plain copy of N bytes fetches N and writes N: scale KiB readings to bytes
    sf = a.copy_bytes / (med(cfetch) * 1024.0)
    sw = a.copy_bytes / (med(cwrite) * 1024.0)
    fb = med(fetch) * 1024.0 * sf
    wb = med(write) * 1024.0 * sw
    lines = [f"# HBM traffic per launch: {a.title}",
             f"command_fetch = {a.command_fetch}",
             f"command_write = {a.command_write}",
             f"command_copy = {a.command_copy}",
             f"kernel = {a.kernel}",
             f"grid_size = {a.grid_size}",
             f"kernel_source = {a.source}",
             f"kernel_source_sha256 = {source_hash(a.source)}",
             f"dispatches = {len(fetch)}",
             f"fetch_kib_median = {med(fetch):.1f}",
             f"write_kib_median = {med(write):.1f}",
             f"copy_bytes = {a.copy_bytes}",
             f"copy_fetch_kib_median = {med(cfetch):.1f}",
             f"copy_write_kib_median = {med(cwrite):.1f}",
             f"fetch_scale = {sf:.4f}",
             f"write_scale = {sw:.4f}",
             f"fetch_bytes_per_launch = {fb:.0f}",
             f"write_bytes_per_launch = {wb:.0f}",
             f"traffic_bytes_per_launch = {fb + wb:.0f}"]
    _write(a.out, lines)


def read_summary(path: str) -> Dict[str, str]:
    d: Dict[str, str] = {}
    with open(path) as f:
        for ln in f:
            if "=" in ln and not ln.lstrip().startswith("#"):
                k, v = ln.split("=", 1)
                d[k.strip()] = v.strip()
    return d


def traffic_if_current(summary: str, root: str) -> Optional[float]:
    """Bytes per launch from a traffic summary, or None if the summary is
    missing or the kernel source changed since the counters were taken."""
    if not os.path.exists(summary):
        return None
    d = read_summary(summary)
    src = os.path.join(root, d.get("kernel_source", ""))
    if not os.path.exists(src) or source_hash(src) != d.get("kernel_source_sha256"):
        return None
    try:
        return float(d["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _write(path: str, lines: List[str]) -> None:
    with open(path, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def main() -> None:
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    s = sub.add_parser("stats")
    s.add_argument("stats_csv")
    s.add_argument("--out", required=True)
    s.add_argument("--title", required=True)
    s.add_argument("--command", required=True)
    s.add_argument("--kernel", nargs="*")
    s.add_argument("--trace", default=None, help="the run's *_kernel_trace.csv")
    t = sub.add_parser("traffic")
    for k in ("fetch_csv", "write_csv", "copy_fetch_csv", "copy_write_csv"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    t.add_argument("--kernel", required=True)
    t.add_argument("--grid-size", type=int, default=None)
    t.add_argument("--copy-kernel", default="elementwise")
    t.add_argument("--copy-bytes", type=int, required=True)
    t.add_argument("--source", required=True)
    t.add_argument("--out", required=True)
    t.add_argument("--title", required=True)
    for k in ("command_fetch", "command_write", "command_copy"):
        t.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    a = ap.parse_args()
    {"stats": cmd_stats, "traffic": cmd_traffic}[a.cmd](a)


if __name__ == "__main__":
    main()
