"""Summarise rocprofv3 CSV output (kernel stats and --pmc counter collections) as short text.

    python -m paper_2606_21238_amd.profsum <rocprofv3 -d directory> [--match REGEX]

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


if __name__ == "__main__":
    args = sys.argv[1:]
    m = None
    if "--match" in args:
        i = args.index("--match")
        m = args[i + 1]
        del args[i:i + 2]
    sys.stdout.write(summarize(args[0], m))
