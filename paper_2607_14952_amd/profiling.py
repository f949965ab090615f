"""Summaries of rocprofv3 output (kernel statistics and byte counters).

Usage:
  python -m paper_2607_14952_amd.profiling stats <rocprof dir> <out.md> --command "..."
  python -m paper_2607_14952_amd.profiling util <rocprof --pmc dir> <out.md> --command "..."
  python -m paper_2607_14952_amd.profiling traffic <FETCH_SIZE dir> <WRITE_SIZE dir> <out.json>
         --calib-bytes N --command "..."

`traffic` scales each kernel's per-dispatch FETCH_SIZE / WRITE_SIZE by what the
same counter reads for the calibration copy kernel of known size, and records
a hash of the kernel sources so that stale counters are not reported.
"""
from __future__ import annotations

import argparse
import csv
import glob
import hashlib
import json
import os
from collections import defaultdict

CSRC = os.path.join(os.path.dirname(os.path.abspath(__file__)), "csrc")
COPY_KERNEL_HINT = "copy"


def source_hash() -> str:
    h = hashlib.sha256()
    for path in sorted(glob.glob(os.path.join(CSRC, "*"))):
        if path.endswith((".hip", ".h", ".cpp")):
            h.update(os.path.basename(path).encode())
            with open(path, "rb") as f:
                h.update(f.read())
    return h.hexdigest()[:16]


def _median(xs):
    if not xs:
        return None
    ys = sorted(xs)
    n = len(ys)
    return ys[n // 2] if n % 2 else 0.5 * (ys[n // 2 - 1] + ys[n // 2])


def _find(directory: str, suffix: str):
    return sorted(glob.glob(os.path.join(directory, "**", f"*{suffix}"), recursive=True))


def _col(row: dict, *names):
    for n in names:
        if n in row and row[n] != "":
            return row[n]
    raise KeyError(f"none of {names} in {list(row)}")


def kernel_stats(directory: str):
    files = _find(directory, "kernel_stats.csv")
    if not files:
        raise FileNotFoundError(f"no kernel_stats.csv under {directory}")
    out = []
    with open(files[0]) as f:
        for row in csv.DictReader(f):
            out.append(dict(name=_col(row, "Name", "KernelName", "Kernel_Name"),
                            calls=int(_col(row, "Calls")),
                            total_ns=float(_col(row, "TotalDurationNs")),
                            avg_ns=float(_col(row, "AverageNs")),
                            min_ns=float(_col(row, "MinNs")),
                            max_ns=float(_col(row, "MaxNs")),
                            pct=float(_col(row, "Percentage"))))
    return out


def dispatch_durations(directory: str):
    """kernel name -> list of dispatch durations (ns) from the kernel trace."""
    files = _find(directory, "kernel_trace.csv")
    if not files:
        return {}
    per = defaultdict(list)
    with open(files[0]) as f:
        for row in csv.DictReader(f):
            name = _col(row, "Kernel_Name", "KernelName", "Name")
            t = float(_col(row, "End_Timestamp")) - float(_col(row, "Start_Timestamp"))
            per[name].append(t)
    return per


def dispatch_medians(directory: str):
    """kernel name -> median dispatch duration (ns) from the kernel trace."""
    return {k: _median(v) for k, v in dispatch_durations(directory).items()}


def long_launches(durations, min_ms: float = 1.0):
    """For a kernel launched at very different sizes (its shortest dispatch
    under a fifth of its longest, the longest at least min_ms), the count and
    mean duration (ns) of the dispatches at least half as long as the longest;
    None otherwise."""
    if not durations:
        return None
    hi = max(durations)
    if hi < min_ms * 1e6 or min(durations) >= 0.2 * hi:
        return None
    big = [d for d in durations if d >= 0.5 * hi]
    return len(big), sum(big) / len(big)


def write_stats_md(directory: str, out_path: str, command: str, title: str) -> None:
    rows = kernel_stats(directory)
    med = dispatch_medians(directory)
    lines = [f"# {title}", "", "Command (run from the repository root on one MI355X):", "",
             "```", command, "```", "",
             f"Kernel sources: `{source_hash()}` (sha256/16 of `paper_2607_14952_amd/csrc`).", "",
             "| kernel | calls | avg ms | median ms | min ms | max ms | total ms | % |",
             "|---|---:|---:|---:|---:|---:|---:|---:|"]
    for r in sorted(rows, key=lambda r: -r["total_ns"]):
        m = med.get(r["name"])
        ms = f"{m / 1e6:.3f}" if m is not None else "-"
        lines.append(f"| `{r['name'][:110]}` | {r['calls']} | {r['avg_ns'] / 1e6:.3f} | {ms} | "
                     f"{r['min_ns'] / 1e6:.3f} | {r['max_ns'] / 1e6:.3f} | "
                     f"{r['total_ns'] / 1e6:.2f} | {r['pct']:.2f} |")
    durs = dispatch_durations(directory)
    mixed = []
    for r in sorted(rows, key=lambda r: -r["total_ns"]):
        ll = long_launches(durs.get(r["name"], []))
        if ll is not None:
            mixed.append(f"| `{r['name'][:110]}` | {ll[0]} | {ll[1] / 1e6:.3f} |")
    if mixed:
        lines += ["", "Kernels launched at very different sizes (for example one call per prefix "
                  "shard and a short one over the response keys): count and mean duration of "
                  "the launches at least half as long as the longest.", "",
                  "| kernel | long launches | avg ms |", "|---|---:|---:|"] + mixed
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")


def counter_per_dispatch(directory: str, counter: str):
    """kernel name -> list of per-dispatch counter values."""
    files = _find(directory, "counter_collection.csv")
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {directory}")
    per = defaultdict(float)
    names = {}
    with open(files[0]) as f:
        for row in csv.DictReader(f):
            if _col(row, "Counter_Name", "CounterName") != counter:
                continue
            d = _col(row, "Dispatch_Id", "DispatchId", "Correlation_Id")
            per[d] += float(_col(row, "Counter_Value", "CounterValue"))
            names[d] = _col(row, "Kernel_Name", "KernelName", "Name")
    out = defaultdict(list)
    for d, v in per.items():
        out[names[d]].append(v)
    return out


UTIL_COUNTERS = ["SQ_INSTS_VALU_MFMA_MOPS_BF16", "SQ_VALU_MFMA_BUSY_CYCLES", "GRBM_GUI_ACTIVE",
                 "SQ_BUSY_CYCLES", "SQ_LDS_IDX_ACTIVE", "SQ_LDS_BANK_CONFLICT"]
N_XCD, N_CU, N_SIMD = 8, 256, 1024


def write_util_md(directory: str, out_path: str, command: str, title: str,
                  min_ms: float = 1.0) -> None:
    """Per kernel (median over its dispatches longer than min_ms): the clock
    (GRBM_GUI_ACTIVE, one count per XCD, over the dispatch time), MFMA-busy
    share of SIMD cycles, executed bf16 MFMA work (MOPS x 512 flop) and its
    rate, LDS-active and bank-conflict shares of CU cycles."""
    files = _find(directory, "counter_collection.csv")
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {directory}")
    disp = defaultdict(dict)
    meta = {}
    with open(files[0]) as f:
        for row in csv.DictReader(f):
            d = _col(row, "Dispatch_Id", "DispatchId", "Correlation_Id")
            c = _col(row, "Counter_Name", "CounterName")
            disp[d][c] = disp[d].get(c, 0.0) + float(_col(row, "Counter_Value", "CounterValue"))
            ns = int(_col(row, "End_Timestamp", "EndTimestamp")) - int(
                _col(row, "Start_Timestamp", "StartTimestamp"))
            meta[d] = (_col(row, "Kernel_Name", "KernelName", "Name"), ns)
    per = defaultdict(list)
    for d, c in disp.items():
        name, ns = meta[d]
        if ns / 1e6 >= min_ms and "GRBM_GUI_ACTIVE" in c:
            per[name].append((ns, c))
    lines = [f"# {title}", "", "Command (run from the repository root on one MI355X):", "",
             "```", command, "```", "",
             f"Kernel sources: `{source_hash()}` (sha256/16 of `paper_2607_14952_amd/csrc`).", "",
             "Per kernel, the dispatch with the median duration among those longer than "
             f"{min_ms} ms. The clock is GRBM_GUI_ACTIVE / {N_XCD} XCDs / duration. MFMA busy is "
             f"SQ_VALU_MFMA_BUSY_CYCLES / ({N_SIMD} SIMDs x GUI cycles). Executed bf16 work is "
             "SQ_INSTS_VALU_MFMA_MOPS_BF16 x 512 flop. LDS active and bank conflict are "
             f"SQ_LDS_IDX_ACTIVE and SQ_LDS_BANK_CONFLICT / ({N_CU} CUs x GUI cycles). The "
             "2.5 PFLOP/s peak assumes 2.4 GHz; 'peak at clock' scales it to the measured clock.",
             "", "| kernel | dispatches | ms | clock GHz | MFMA busy % | executed TFLOP | "
             "executed TFLOP/s | % of peak at clock | LDS active % | bank conflict % |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for name, lst in sorted(per.items(), key=lambda kv: -sum(ns for ns, _ in kv[1])):
        lst.sort(key=lambda t: t[0])
        ns, c = lst[len(lst) // 2]
        gui = c["GRBM_GUI_ACTIVE"] / N_XCD
        clk = gui / ns
        busy = 100 * c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0) / (N_SIMD * gui)
        fl = c.get("SQ_INSTS_VALU_MFMA_MOPS_BF16", 0) * 512
        rate = fl / (ns * 1e-9) / 1e12
        peak_clk = 2500.0 * clk / 2.4
        lds = 100 * c.get("SQ_LDS_IDX_ACTIVE", 0) / (N_CU * gui)
        bank = 100 * c.get("SQ_LDS_BANK_CONFLICT", 0) / (N_CU * gui)
        lines.append(f"| `{name[:90]}` | {len(lst)} | {ns / 1e6:.3f} | {clk:.2f} | {busy:.1f} | "
                     f"{fl / 1e12:.2f} | {rate:.0f} | {100 * rate / peak_clk:.1f} | {lds:.1f} | "
                     f"{bank:.2f} |")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")


WAIT_COUNTERS = ["SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY",
                 "SQ_ACTIVE_INST_VALU", "SQ_INSTS_VALU", "SQ_INSTS_LDS", "SQ_WAIT_INST_LDS"]


def write_waits_md(directory: str, out_path: str, command: str, title: str,
                   min_ms: float = 1.0) -> None:
    """Per kernel (median dispatch longer than min_ms): where the waves' cycles
    go, as shares of SQ_WAVE_CYCLES (issuing any instruction, issuing VALU
    instructions, waiting on a counter before the next instruction, waiting at
    all), and the VALU and LDS instructions per dispatch."""
    files = _find(directory, "counter_collection.csv")
    if not files:
        raise FileNotFoundError(f"no counter_collection.csv under {directory}")
    disp = defaultdict(dict)
    meta = {}
    with open(files[0]) as f:
        for row in csv.DictReader(f):
            d = _col(row, "Dispatch_Id", "DispatchId", "Correlation_Id")
            c = _col(row, "Counter_Name", "CounterName")
            disp[d][c] = disp[d].get(c, 0.0) + float(_col(row, "Counter_Value", "CounterValue"))
            ns = int(_col(row, "End_Timestamp", "EndTimestamp")) - int(
                _col(row, "Start_Timestamp", "StartTimestamp"))
            meta[d] = (_col(row, "Kernel_Name", "KernelName", "Name"), ns)
    per = defaultdict(list)
    for d, c in disp.items():
        name, ns = meta[d]
        if ns / 1e6 >= min_ms and c.get("SQ_WAVE_CYCLES"):
            per[name].append((ns, c))
    lines = [f"# {title}", "", "Command (run from the repository root on one MI355X):", "",
             "```", command, "```", "",
             f"Kernel sources: `{source_hash()}` (sha256/16 of `paper_2607_14952_amd/csrc`).", "",
             f"Per kernel, the dispatch with the median duration among those longer than {min_ms} "
             "ms. Shares are of SQ_WAVE_CYCLES: issuing any instruction (SQ_ACTIVE_INST_ANY), "
             "issuing VALU instructions including MFMAs (SQ_ACTIVE_INST_VALU), waiting for a "
             "counter before the next instruction (SQ_WAIT_INST_ANY), waiting at all (SQ_WAIT_ANY), "
             "and waiting for LDS (SQ_WAIT_INST_LDS).", "",
             "| kernel | ms | issue any % | issue VALU % | wait for counter % | wait any % | "
             "wait LDS % | VALU instructions | LDS instructions |",
             "|---|---:|---:|---:|---:|---:|---:|---:|---:|"]
    for name, lst in sorted(per.items(), key=lambda kv: -sum(ns for ns, _ in kv[1])):
        lst.sort(key=lambda t: t[0])
        ns, c = lst[len(lst) // 2]
        wc = c["SQ_WAVE_CYCLES"]
        pct = lambda k: 100 * c.get(k, 0) / wc  # noqa: E731
        lines.append(f"| `{name[:90]}` | {ns / 1e6:.3f} | {pct('SQ_ACTIVE_INST_ANY'):.1f} | "
                     f"{pct('SQ_ACTIVE_INST_VALU'):.1f} | {pct('SQ_WAIT_INST_ANY'):.1f} | "
                     f"{pct('SQ_WAIT_ANY'):.1f} | {pct('SQ_WAIT_INST_LDS'):.1f} | "
                     f"{c.get('SQ_INSTS_VALU', 0):.3g} | {c.get('SQ_INSTS_LDS', 0):.3g} |")
    with open(out_path, "w") as f:
        f.write("\n".join(lines) + "\n")


def write_traffic(fetch_dir: str, write_dir: str, out_path: str, calib_bytes: int,
                  command: str) -> dict:
    fetch = counter_per_dispatch(fetch_dir, "FETCH_SIZE")
    write = counter_per_dispatch(write_dir, "WRITE_SIZE")

    # The calibration copy is the copy dispatch whose WRITE_SIZE is closest to
    # calib_bytes (the write counter reads copies exactly); the FETCH run
    # dispatches the same kernels in the same order, so the same index is used.
    def copies(per):
        c = [(k, v) for k, v in per.items() if COPY_KERNEL_HINT in k.lower()]
        if not c:
            raise RuntimeError("calibration copy kernel not found in the counter output")
        return c[0]

    ck_w, wv = copies(write)
    ck_f, fv = copies(fetch)
    j = min(range(len(wv)), key=lambda i: abs(wv[i] * 1024.0 - calib_bytes))
    if j >= len(fv):
        raise RuntimeError("the FETCH run has fewer copy dispatches than the WRITE run")
    cf, cw = fv[j], wv[j]
    scale_f = calib_bytes / (cf * 1024.0)
    scale_w = calib_bytes / (cw * 1024.0)
    kernels = {}
    for name in sorted(set(fetch) | set(write)):
        f = fetch.get(name, [])
        w = write.get(name, [])
        mf, mw = _median(f), _median(w)
        kernels[name] = {
            "dispatches": max(len(f), len(w)),
            "fetch_kib_per_dispatch_median": mf,
            "write_kib_per_dispatch_median": mw,
            "fetch_kib_per_dispatch": f,
            "write_kib_per_dispatch": w,
            "hbm_bytes_per_dispatch": (mf or 0.0) * 1024 * scale_f + (mw or 0.0) * 1024 * scale_w,
        }
    doc = {"command": command, "source_hash": source_hash(), "calib_bytes": calib_bytes,
           "calib_kernel": {"fetch": ck_f, "write": ck_w},
           "calib_counter_kib": {"FETCH_SIZE": cf, "WRITE_SIZE": cw},
           "scale": {"FETCH_SIZE": scale_f, "WRITE_SIZE": scale_w}, "kernels": kernels}
    with open(out_path, "w") as fo:
        json.dump(doc, fo, indent=1)
    return doc


def traffic_for(kernel_substr: str, path: str):
    """HBM bytes per dispatch of the first kernel matching kernel_substr, or None
    when the file is missing or was taken from other kernel sources."""
    if not os.path.exists(path):
        return None
    with open(path) as f:
        doc = json.load(f)
    if doc.get("source_hash") != source_hash():
        return None
    for name, v in doc["kernels"].items():
        if kernel_substr in name:
            return v["hbm_bytes_per_dispatch"]
    return None


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("directory")
    a.add_argument("out")
    a.add_argument("--command", required=True)
    a.add_argument("--title", default="rocprofv3 kernel statistics")
    u = sub.add_parser("util")
    u.add_argument("directory")
    u.add_argument("out")
    u.add_argument("--command", required=True)
    u.add_argument("--title", default="rocprofv3 MFMA and LDS utilization")
    u.add_argument("--min-ms", type=float, default=1.0)
    wt = sub.add_parser("waits")
    wt.add_argument("directory")
    wt.add_argument("out")
    wt.add_argument("--command", required=True)
    wt.add_argument("--title", default="rocprofv3 issue and wait counters")
    wt.add_argument("--min-ms", type=float, default=1.0)
    b = sub.add_parser("traffic")
    b.add_argument("fetch_dir")
    b.add_argument("write_dir")
    b.add_argument("out")
    b.add_argument("--calib-bytes", type=int, required=True)
    b.add_argument("--command", required=True)
    args = ap.parse_args()
    if args.cmd == "stats":
        write_stats_md(args.directory, args.out, args.command, args.title)
    elif args.cmd == "util":
        write_util_md(args.directory, args.out, args.command, args.title, args.min_ms)
    elif args.cmd == "waits":
        write_waits_md(args.directory, args.out, args.command, args.title, args.min_ms)
    else:
        write_traffic(args.fetch_dir, args.write_dir, args.out, args.calib_bytes, args.command)


if __name__ == "__main__":
    main()
