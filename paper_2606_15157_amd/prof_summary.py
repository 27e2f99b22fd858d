"""Markdown table of per-kernel durations from a rocprofv3 --kernel-trace --stats run.

    rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -o run -- python3 bench.py \
        --steps 50 --warmup 5 --no-cpu-baseline
    python -m paper_2606_15157_amd.prof_summary <dir> <out.md> "<title>" "<command>" \
        [<kernel> <skip> <n>]

With <kernel>, <skip> and <n>, dispatches skip .. skip + n - 1 of that kernel (by start time;
in the default benchmark run, after the 100 settle and 5 warm-up passes, these are the 50 timed
passes of the headline route) are also averaged on their own from the kernel trace.
"""
from __future__ import annotations

import csv
import glob
import os
import re
import sys


def kernel_stats(run_dir: str):
    path = glob.glob(os.path.join(run_dir, "**", "*kernel_stats.csv"), recursive=True)
    if not path:
        raise FileNotFoundError(f"no kernel_stats.csv under {run_dir}")
    rows = list(csv.DictReader(open(path[0])))
    return sorted(rows, key=lambda r: -float(r["TotalDurationNs"]))


def short_name(name: str) -> str:
    """Kernel name without return type, namespaces and parameter list."""
    name = re.sub(r"^void ", "", name)
    if name.startswith("at::"):   # torch's own kernels (input generation in the benchmark)
        return "torch " + re.split(r"[<(]", name)[0]
    name = name.replace("rkv::(anonymous namespace)::", "")
    depth, cut = 0, len(name)
    for i, ch in enumerate(name):      # drop the parameter list: the first '(' outside <...>
        depth += (ch == "<") - (ch == ">")
        if ch == "(" and depth == 0:
            cut = i
            break
    return name[:cut]


def dispatches(run_dir: str, kernel: str, skip: int, n: int):
    """Durations (ns) of the first n dispatches of the kernel whose short name is `kernel`."""
    path = glob.glob(os.path.join(run_dir, "**", "*kernel_trace.csv"), recursive=True)
    if not path:
        raise FileNotFoundError(f"no kernel_trace.csv under {run_dir}")
    rows = [r for r in csv.DictReader(open(path[0])) if short_name(r["Kernel_Name"]) == kernel]
    rows.sort(key=lambda r: int(r["Start_Timestamp"]))
    return [int(r["End_Timestamp"]) - int(r["Start_Timestamp"]) for r in rows[skip:skip + n]]


MAX_ROWS = 25   # the table lists the kernels with the largest total time


def main(argv):
    run_dir, out_md, title, command = argv[1:5]
    rows = kernel_stats(run_dir)
    with open(out_md, "w") as f:
        f.write(f"# {title}\n\nCommand (from /tmp with TMPDIR=/tmp):\n\n    {command}\n\n")
        f.write("| kernel | calls | average (us) | min (us) | max (us) | share |\n|---|---|---|---|---|---|\n")
        for r in rows[:MAX_ROWS]:
            f.write(f"| {short_name(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                    f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                    f"{float(r['Percentage']):.1f}% |\n")
        if len(rows) > MAX_ROWS:
            rest = sum(float(r["Percentage"]) for r in rows[MAX_ROWS:])
            f.write(f"| ({len(rows) - MAX_ROWS} more kernels) | | | | | {rest:.1f}% |\n")
        if len(argv) > 7:
            kernel, skip, n = argv[5], int(argv[6]), int(argv[7])
            d = dispatches(run_dir, kernel, skip, n)
            f.write(f"\nDispatches {skip}-{skip + len(d) - 1} of {kernel} (the headline route's timed passes): "
                    f"average {sum(d) / len(d) / 1e3:.1f} us, min {min(d) / 1e3:.1f} us, "
                    f"max {max(d) / 1e3:.1f} us.\n")
    print(open(out_md).read())


if __name__ == "__main__":
    main(sys.argv)
