"""Kernel-duration statistics of a workload in the form of the paper's
micro-kernel table (section 2.4, table of kernel durations after graph
capture): the median kernel duration in cycles and the share of kernels
shorter than 5K, 10K, 25K and 50K cycles.

    python paper_2609_22335_amd/trace_stats.py --clock-ghz 2.4 \
        vlm=<vlm kernel_trace.csv> action=<action kernel_trace.csv>

Each argument is a phase name and a rocprofv3 `--kernel-trace -f csv` file of
that phase run on its own (profile_intensity.py --run vlm|action makes such
runs). Durations are End - Start timestamps (ns) converted to cycles at the
given clock; the table has one row per phase and one for all kernels.
Kernels whose name matches --skip (set-up copies, weight re-layout) are left
out.
"""
from __future__ import annotations

import argparse
import csv
import re
from typing import Dict, Iterable, List, Sequence

BUCKETS = (5_000, 10_000, 25_000, 50_000)
DEFAULT_SKIP = r"k_unfrag|k_copy|elementwise|fill|copy_kernel"


def durations_ns(path: str, skip: str = DEFAULT_SKIP) -> List[int]:
    """Kernel durations (ns) of a rocprofv3 kernel trace, in trace order."""
    pat = re.compile(skip) if skip else None
    out = []
    with open(path, newline="") as f:
        for r in csv.DictReader(f):
            if pat and pat.search(r["Kernel_Name"]):
                continue
            out.append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    return out


def median(xs: Sequence[float]) -> float:
    s = sorted(xs)
    n = len(s)
    if n == 0:
        raise ValueError("no kernels")
    return float(s[n // 2]) if n % 2 else 0.5 * (s[n // 2 - 1] + s[n // 2])


def table_row(dur_ns: Iterable[float], clock_ghz: float) -> Dict[str, float]:
    """Median duration in cycles and the percentage of kernels below each
    bucket bound (strictly shorter), for durations in ns."""
    cyc = [d * clock_ghz for d in dur_ns]
    row = {"kernels": len(cyc), "median_cyc": median(cyc)}
    for b in BUCKETS:
        row[f"lt{b // 1000}k_pct"] = 100.0 * sum(c < b for c in cyc) / len(cyc)
    return row


def markdown(rows: Dict[str, Dict[str, float]], clock_ghz: float) -> str:
    lines = [f"| phase | kernels | median (cyc) | <5K % | <10K % | <25K % | <50K % |",
             "|---|---|---|---|---|---|---|"]
    for name, r in rows.items():
        lines.append(f"| {name} | {r['kernels']} | {r['median_cyc']:.0f} | {r['lt5k_pct']:.1f} | "
                     f"{r['lt10k_pct']:.1f} | {r['lt25k_pct']:.1f} | {r['lt50k_pct']:.1f} |")
    lines.append(f"\nCycles = trace duration (ns) x {clock_ghz} GHz.")
    return "\n".join(lines)


def main(argv=None) -> None:
    ap = argparse.ArgumentParser()
    ap.add_argument("--clock-ghz", type=float, default=2.4)
    ap.add_argument("--skip", default=DEFAULT_SKIP)
    ap.add_argument("phases", nargs="+", help="name=kernel_trace.csv")
    a = ap.parse_args(argv)
    rows, allv = {}, []
    for item in a.phases:
        name, path = item.split("=", 1)
        d = durations_ns(path, a.skip)
        rows[name] = table_row(d, a.clock_ghz)
        allv += d
    if len(a.phases) > 1:
        rows["all"] = table_row(allv, a.clock_ghz)
    print(markdown(rows, a.clock_ghz))


if __name__ == "__main__":
    main()
