"""Turn rocprofv3 CSV output into the short text summaries kept in profiles/.

``stats``: per-kernel call count and average / total duration from a
``--kernel-trace --stats`` run; with ``--trace`` the per-dispatch trace of the
same run is split by grid size, so that launches of one kernel on different
workloads are averaged apart. ``traffic-req``: HBM bytes per launch of one
kernel from the L2's memory-request counts by request size (two ``--pmc``
runs), with a plain copy of known size alongside as a check (not a scale).
``traffic``: the older form, FETCH_SIZE / WRITE_SIZE scaled by what a plain
copy reads. ``mfma``: MFMA utilisation and instruction mix of a bf16 matrix
kernel from three SQ counter passes. Every summary records a hash of the
kernel's source so that a reader can tell whether the counters still
describe the code.

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


RD = ("TCC_EA0_RDREQ_sum", "TCC_EA0_RDREQ_32B_sum", "TCC_EA0_RDREQ_64B_sum",
      "TCC_EA0_RDREQ_128B_sum")
WR = ("TCC_EA0_WRREQ_sum", "TCC_EA0_WRREQ_64B_sum")


def counters_per_dispatch(csv_path: str, kernel_substr: str, names,
                          grid_size: Optional[int] = None) -> List[Dict[str, float]]:
    """{counter: value} per dispatch of the matching kernel (values summed over
    the rows of a dispatch)."""
    per: Dict[str, Dict[str, float]] = {}
    for r in _rows(csv_path):
        name = _col(r, "Kernel_Name", "Kernel-Name", "KernelName") or ""
        cname = _col(r, "Counter_Name", "Counter-Name", "CounterName") or ""
        if kernel_substr not in name or cname not in names:
            continue
        if grid_size is not None and int(float(_col(r, "Grid_Size") or -1)) != grid_size:
            continue
        did = _col(r, "Dispatch_Id", "Dispatch-Id", "DispatchId") or "0"
        d = per.setdefault(did, {})
        d[cname] = d.get(cname, 0.0) + float(_col(r, "Counter_Value", "Counter-Value",
                                                  "CounterValue") or 0.0)
    return [v for v in per.values() if all(n in v for n in names)]


def request_bytes(rd: Dict[str, float], wr: Dict[str, float]):
    """HBM bytes from the L2's memory-request counts by size: reads are 32, 64
    or 128 bytes each, writes 64 bytes or else 32. Returns (read bytes, write
    bytes, read requests of no listed size)."""
    n, n32, n64, n128 = (rd[k] for k in RD)
    read = 32 * n32 + 64 * n64 + 128 * n128
    w, w64 = (wr[k] for k in WR)
    write = 64 * w64 + 32 * (w - w64)
    return read, write, n - n32 - n64 - n128


def cmd_traffic_req(a) -> None:
    med = statistics.median
    rd = counters_per_dispatch(a.rd_csv, a.kernel, RD, a.grid_size)
    wr = counters_per_dispatch(a.wr_csv, a.kernel, WR, a.grid_size)
    crd = counters_per_dispatch(a.copy_rd_csv, a.copy_kernel, RD)
    cwr = counters_per_dispatch(a.copy_wr_csv, a.copy_kernel, WR)
    if not (rd and wr and crd and cwr):
        raise SystemExit(f"missing counter rows: {len(rd)} {len(wr)} {len(crd)} {len(cwr)}")
    m_rd = {k: med(d[k] for d in rd) for k in RD}
    m_wr = {k: med(d[k] for d in wr) for k in WR}
    c_rd = {k: med(d[k] for d in crd) for k in RD}
    c_wr = {k: med(d[k] for d in cwr) for k in WR}
    r, w, unl = request_bytes(m_rd, m_wr)
    cr, cw, cunl = request_bytes(c_rd, c_wr)
    lines = [f"# HBM traffic per launch from L2 memory-request counts: {a.title}",
             f"command_read = {a.command_rd}",
             f"command_write = {a.command_wr}",
             f"command_copy = {a.command_copy}",
             f"kernel = {a.kernel}",
             f"grid_size = {a.grid_size}",
             f"kernel_source = {a.source}",
             f"kernel_source_sha256 = {source_hash(a.source)}",
             f"dispatches = {len(rd)} read, {len(wr)} write",
             "# bytes = 32 x RDREQ_32B + 64 x RDREQ_64B + 128 x RDREQ_128B (reads);",
             "#         64 x WRREQ_64B + 32 x (WRREQ - WRREQ_64B) (writes); no scale factor"]
    lines += [f"{k} = {v:.0f}" for k, v in m_rd.items()]
    lines += [f"{k} = {v:.0f}" for k, v in m_wr.items()]
    lines += [f"read_requests_of_no_listed_size = {unl:.0f}",
              f"check_copy_bytes = {a.copy_bytes}",
              f"check_copy_read_bytes = {cr:.0f}",
              f"check_copy_write_bytes = {cw:.0f}",
              f"check_copy_read_over_known = {cr / a.copy_bytes:.4f}",
              f"check_copy_write_over_known = {cw / a.copy_bytes:.4f}",
              f"read_bytes_per_launch = {r:.0f}",
              f"write_bytes_per_launch = {w:.0f}",
              f"traffic_bytes_per_launch = {r + w:.0f}"]
    if a.algorithmic_bytes:
        lines.append(f"algorithmic_bytes_per_launch = {a.algorithmic_bytes}")
        lines.append(f"traffic_over_algorithmic = {(r + w) / a.algorithmic_bytes:.4f}")
    _write(a.out, lines)


SQ_PASSES = {
    "a": ("SQ_BUSY_CYCLES", "SQ_BUSY_CU_CYCLES", "SQ_VALU_MFMA_BUSY_CYCLES",
          "SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_INSTS_MFMA", "SQ_INSTS_VALU", "SQ_INSTS_SALU",
          "SQ_INSTS_VALU_TRANS_F32"),
    "b": ("SQ_INSTS_LDS", "SQ_LDS_IDX_ACTIVE", "SQ_LDS_BANK_CONFLICT", "SQ_LDS_DATA_FIFO_FULL",
          "SQ_LDS_CMD_FIFO_FULL", "SQ_WAIT_INST_LDS", "SQ_INSTS_SMEM", "SQ_INSTS_BRANCH"),
    "c": ("SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY",
          "SQ_ACTIVE_INST_VALU", "SQ_ACTIVE_INST_LDS", "SQ_ACTIVE_INST_SCA", "SQ_INSTS_VMEM"),
}


def cmd_mfma(a) -> None:
    """MFMA utilisation of a bf16 matrix kernel from three SQ counter passes."""
    med = statistics.median
    vals: Dict[str, float] = {}
    for tag, path in (("a", a.pass_a), ("b", a.pass_b), ("c", a.pass_c)):
        rows = counters_per_dispatch(path, a.kernel, SQ_PASSES[tag], a.grid_size)
        if not rows:
            raise SystemExit(f"no rows for pass {tag}")
        vals.update({k: med(d[k] for d in rows) for k in SQ_PASSES[tag]})
    mfma = vals["SQ_INSTS_MFMA"]
    busy = vals["SQ_VALU_MFMA_BUSY_CYCLES"]
    # busy fraction of the matrix pipes over the kernel's duration, counted in
    # cycles of the 2.4 GHz clock the peak is quoted at (1024 SIMDs)
    frac_2400 = busy / (4 * a.num_cus * a.kernel_us * 1e-6 * 2.4e9)
    flop_exec = vals["SQ_INSTS_VALU_MFMA_MOPS_BF16"] * 512
    lines = [f"# MFMA utilisation from SQ counters: {a.title}",
             f"command_pass_a = {a.command_a}",
             f"command_pass_b = {a.command_b}",
             f"command_pass_c = {a.command_c}",
             f"kernel = {a.kernel}",
             f"grid_size = {a.grid_size}",
             f"kernel_source = {a.source}",
             f"kernel_source_sha256 = {source_hash(a.source)}",
             "# medians per dispatch, summed over the device"]
    lines += [f"{k} = {v:.6g}" for k, v in vals.items()]
    lines += [
        f"kernel_us = {a.kernel_us}",
        f"algorithmic_flop = {a.algorithmic_flop}",
        f"mfma_flop_executed = {flop_exec:.6g}",
        f"mfma_flop_executed_over_algorithmic = {flop_exec / a.algorithmic_flop:.4f}",
        f"mfma_busy_cycles_per_mfma = {busy / mfma:.2f}",
        f"mfma_busy_frac_of_2400mhz_cycles = {frac_2400:.4f}",
        f"tflops_frac_of_2400mhz_peak = {a.algorithmic_flop / (a.kernel_us * 1e-6) / 2516.6e12:.4f}",
    ]
    if a.clock_ghz:
        lines += [f"shader_clock_ghz_measured = {a.clock_ghz}",
                  f"mfma_busy_frac_of_measured_cycles = {frac_2400 * 2.4 / a.clock_ghz:.4f}"]
    lines += [
        f"valu_non_mfma_per_mfma = {(vals['SQ_INSTS_VALU'] - mfma) / mfma:.3f}",
        f"trans_per_mfma = {vals['SQ_INSTS_VALU_TRANS_F32'] / mfma:.3f}",
        f"salu_per_mfma = {vals['SQ_INSTS_SALU'] / mfma:.3f}",
        f"smem_per_mfma = {vals['SQ_INSTS_SMEM'] / mfma:.3f}",
        f"lds_per_mfma = {vals['SQ_INSTS_LDS'] / mfma:.3f}",
        f"branch_per_mfma = {vals['SQ_INSTS_BRANCH'] / mfma:.3f}",
        f"vmem_per_mfma = {vals['SQ_INSTS_VMEM'] / mfma:.4f}",
    ]
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
    r = sub.add_parser("traffic-req")
    for k in ("rd_csv", "wr_csv", "copy_rd_csv", "copy_wr_csv"):
        r.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    r.add_argument("--kernel", required=True)
    r.add_argument("--grid-size", type=int, default=None)
    r.add_argument("--copy-kernel", default="elementwise")
    r.add_argument("--copy-bytes", type=int, required=True)
    r.add_argument("--algorithmic-bytes", type=int, default=None)
    r.add_argument("--source", required=True)
    r.add_argument("--out", required=True)
    r.add_argument("--title", required=True)
    for k in ("command_rd", "command_wr", "command_copy"):
        r.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    m = sub.add_parser("mfma")
    for k in ("pass_a", "pass_b", "pass_c"):
        m.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    m.add_argument("--kernel", required=True)
    m.add_argument("--grid-size", type=int, default=None)
    m.add_argument("--kernel-us", type=float, required=True,
                   help="the kernel's average duration from a --kernel-trace --stats run")
    m.add_argument("--algorithmic-flop", type=float, required=True)
    m.add_argument("--num-cus", type=int, default=256)
    m.add_argument("--clock-ghz", type=float, default=None,
                   help="shader clock measured during the kernel, if known")
    m.add_argument("--source", required=True)
    m.add_argument("--out", required=True)
    m.add_argument("--title", required=True)
    for k in ("command_a", "command_b", "command_c"):
        m.add_argument("--" + k.replace("_", "-"), dest=k, required=True)
    a = ap.parse_args()
    {"stats": cmd_stats, "traffic": cmd_traffic, "traffic-req": cmd_traffic_req,
     "mfma": cmd_mfma}[a.cmd](a)


if __name__ == "__main__":
    main()
