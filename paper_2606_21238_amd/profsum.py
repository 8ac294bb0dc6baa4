"""Summarise rocprofv3 CSV output (kernel stats and --pmc counter collections) as short text.

    python -m paper_2606_21238_amd.profsum <rocprofv3 -d directory> [--match REGEX]
    python -m paper_2606_21238_amd.profsum <dir> --match REGEX --last K     # timed dispatches
    python -m paper_2606_21238_amd.profsum --traffic-json OUT ...           # see the end of file
    python -m paper_2606_21238_amd.profsum <dir> --match REGEX --counters-last K   # SQ counters

Kernel stats: calls, total and average duration per kernel.  Counter collections: per
kernel and counter, the number of dispatches and the mean value per dispatch.
"""

from __future__ import annotations

import csv
import glob
import os
import re
import sys
from collections import defaultdict


def _short(name: str) -> str:
    name = name.replace("(anonymous namespace)::", "")
    if name.startswith("void "):
        name = name[5:]
    name = re.sub(r"\(.*", "", name)                      # drop the parameter list
    return name[:90]


def _col(row: dict, *cands):
    low = {k.lower(): k for k in row}
    for c in cands:
        if c.lower() in low:
            return row[low[c.lower()]]
    raise KeyError(cands)


def summarize(directory: str, match: str | None = None) -> str:
    out = []
    rx = re.compile(match) if match else None
    for path in sorted(glob.glob(os.path.join(directory, "**", "*kernel_stats.csv"), recursive=True)):
        out.append(f"# kernel stats ({os.path.basename(path)})")
        out.append(f"{'kernel':<90} {'calls':>7} {'total_us':>12} {'avg_us':>10} {'pct':>6}")
        with open(path) as f:
            for row in csv.DictReader(f):
                name = _col(row, "Name", "KernelName", "Kernel_Name")
                if rx and not rx.search(name):
                    continue
                calls = int(float(_col(row, "Calls")))
                total = float(_col(row, "TotalDurationNs", "Total_Duration_Ns")) / 1e3
                avg = float(_col(row, "AverageNs", "Average_Ns")) / 1e3
                pct = float(_col(row, "Percentage"))
                out.append(f"{_short(name):<90} {calls:>7} {total:>12.1f} {avg:>10.2f} {pct:>6.2f}")
    for path in sorted(glob.glob(os.path.join(directory, "**", "*counter_collection.csv"), recursive=True)):
        acc = defaultdict(lambda: [0, 0.0])
        with open(path) as f:
            for row in csv.DictReader(f):
                name = _col(row, "Kernel_Name", "KernelName")
                if rx and not rx.search(name):
                    continue
                key = (_short(name), _col(row, "Counter_Name", "CounterName"))
                acc[key][0] += 1
                acc[key][1] += float(_col(row, "Counter_Value", "CounterValue"))
        out.append(f"# counters per dispatch ({os.path.basename(path)})")
        out.append(f"{'kernel':<90} {'counter':<28} {'dispatches':>10} {'mean':>16}")
        for (k, c), (n, s) in sorted(acc.items()):
            out.append(f"{k:<90} {c:<28} {n:>10} {s / n:>16.1f}")
    return "\n".join(out) + "\n"


def _dispatches(directory: str, kind: str):
    """Rows of the kernel-trace or counter-collection CSVs, in dispatch order."""
    rows = []
    for path in glob.glob(os.path.join(directory, "**", f"*{kind}.csv"), recursive=True):
        with open(path) as f:
            rows += list(csv.DictReader(f))
    key = "Start_Timestamp" if kind == "kernel_trace" else "Dispatch_Id"
    rows.sort(key=lambda r: int(float(_col(r, key))))
    return rows


def last_durations(directory: str, match: str, last: int) -> str:
    """Mean duration of each matching kernel over its last `last` dispatches (the timed steps of
    a bench run come last)."""
    per = defaultdict(list)
    for r in _dispatches(directory, "kernel_trace"):
        name = _col(r, "Kernel_Name", "KernelName")
        if re.search(match, name):
            per[_short(name)].append((int(_col(r, "End_Timestamp")) - int(_col(r, "Start_Timestamp"))) / 1e3)
    out = [f"# mean over the last {last} dispatches (kernel_trace.csv)",
           f"{'kernel':<90} {'dispatches':>10} {'avg_us':>10}"]
    for k, v in sorted(per.items()):
        tail = v[-last:]
        out.append(f"{k:<90} {len(tail):>10} {sum(tail) / len(tail):>10.2f}")
    return "\n".join(out) + "\n"


def last_counter(directory: str, match: str, counter: str, last: int) -> float:
    """Mean value of `counter` per dispatch of the kernels matching `match`, over the last
    `last` such dispatches (values of one dispatch summed over its rows)."""
    per = defaultdict(float)
    order = []
    for r in _dispatches(directory, "counter_collection"):
        name = _col(r, "Kernel_Name", "KernelName")
        if not re.search(match, name) or _col(r, "Counter_Name", "CounterName") != counter:
            continue
        d = int(float(_col(r, "Dispatch_Id")))
        if d not in per:
            order.append(d)
        per[d] += float(_col(r, "Counter_Value", "CounterValue"))
    tail = order[-last:]
    return sum(per[d] for d in tail) / max(1, len(tail))


def counter_names(directory: str, match: str) -> list:
    names = []
    for r in _dispatches(directory, "counter_collection"):
        c = _col(r, "Counter_Name", "CounterName")
        if re.search(match, _col(r, "Kernel_Name", "KernelName")) and c not in names:
            names.append(c)
    return names


def counters_last(directory: str, match: str, last: int, xcds: int = 8, simds: int = 1024) -> str:
    """Mean per dispatch of every counter of the kernels matching `match` over their last
    `last` dispatches, and, when the pass holds them, the MFMA-busy fraction
    SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / xcds * simds): GRBM_GUI_ACTIVE counts the
    dispatch's GPU-active cycles once per XCD, SQ_VALU_MFMA_BUSY_CYCLES the matrix-core busy
    cycles summed over all SIMDs (MI355X: 8 XCDs, 256 CUs x 4 SIMDs)."""
    vals = {c: last_counter(directory, match, c, last) for c in counter_names(directory, match)}
    out = [f"# counters, mean per dispatch over the last {last} dispatches of /{match}/"]
    out += [f"{c:34s} {v:20.1f}" for c, v in vals.items()]
    if "SQ_VALU_MFMA_BUSY_CYCLES" in vals and vals.get("GRBM_GUI_ACTIVE"):
        cyc = vals["GRBM_GUI_ACTIVE"] / xcds
        out.append(f"# active cycles per XCD {cyc:.4g}; MFMA busy fraction "
                   f"{vals['SQ_VALU_MFMA_BUSY_CYCLES'] / (cyc * simds):.4f}")
    if "SQ_INSTS_MFMA" in vals and vals.get("SQ_INSTS_VALU"):
        out.append(f"# non-MFMA VALU instructions per MFMA "
                   f"{(vals['SQ_INSTS_VALU'] - vals['SQ_INSTS_MFMA']) / max(vals['SQ_INSTS_MFMA'], 1):.2f}")
    if "SQ_VALU_MFMA_COEXEC_CYCLES" in vals and vals.get("SQ_VALU_MFMA_BUSY_CYCLES"):
        out.append(f"# VALU issued during MFMA-busy cycles "
                   f"{vals['SQ_VALU_MFMA_COEXEC_CYCLES'] / vals['SQ_VALU_MFMA_BUSY_CYCLES']:.4f}")
    return "\n".join(out) + "\n"


def traffic_entry(fetch_dir: str, write_dir: str, kernel: str, calib: str, calib_mib: int, last: int):
    """HBM bytes per launch of `kernel` from FETCH_SIZE / WRITE_SIZE (KiB per dispatch), each
    scaled by what the counter reads for the calibration kernel that reads and writes exactly
    `calib_mib` MiB."""
    f_cal = last_counter(fetch_dir, calib, "FETCH_SIZE", 1)
    w_cal = last_counter(write_dir, calib, "WRITE_SIZE", 1)
    f_factor = calib_mib * 1024.0 / f_cal
    w_factor = calib_mib * 1024.0 / w_cal
    fetch = last_counter(fetch_dir, kernel, "FETCH_SIZE", last) * 1024.0 * f_factor
    write = last_counter(write_dir, kernel, "WRITE_SIZE", last) * 1024.0 * w_factor
    return {"fetch_bytes_per_launch": fetch, "write_bytes_per_launch": write,
            "fetch_factor": f_factor, "write_factor": w_factor, "dispatches": last}


if __name__ == "__main__":
    args = sys.argv[1:]

    def opt(name, default=None):
        if name in args:
            i = args.index(name)
            v = args[i + 1]
            del args[i:i + 2]
            return v
        return default

    m = opt("--match")
    last = opt("--last")
    traffic = opt("--traffic-json")
    clast = opt("--counters-last")
    if clast:
        sys.stdout.write(counters_last(args[0], m or ".", int(clast)))
    elif traffic:
        # --traffic-json OUT --workload W --kernel-source SRC --fetch-dir D1 --write-dir D2
        #   --calib-match REGEX --calib-mib N --last K --match KERNEL_REGEX [--kernel-name NAME]
        import hashlib
        import json
        w = opt("--workload")
        src = opt("--kernel-source")
        kname = opt("--kernel-name")
        entry = traffic_entry(opt("--fetch-dir"), opt("--write-dir"), m, opt("--calib-match"),
                              int(opt("--calib-mib")), int(last))
        entry["kernel"] = kname or m
        sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
        data = json.load(open(traffic)) if os.path.exists(traffic) else {}
        if data.get("kernel_source_sha256") != sha:
            data = {"kernel_source_sha256": sha, "workloads": {}}
        data["workloads"][w] = entry
        json.dump(data, open(traffic, "w"), indent=1, sort_keys=True)
        print(json.dumps({w: entry}))
    elif last:
        sys.stdout.write(last_durations(args[0], m or ".", int(last)))
    else:
        sys.stdout.write(summarize(args[0], m))
