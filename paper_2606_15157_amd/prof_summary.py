"""Markdown table of per-kernel durations from a rocprofv3 --kernel-trace --stats run.

    rocprofv3 --kernel-trace --stats --output-format csv -d <dir> -o run -- python3 bench.py \
        --steps 50 --warmup 5 --no-cpu-baseline
    python -m paper_2606_15157_amd.prof_summary <dir> <out.md> "<title>" "<command>"
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


def main(argv):
    run_dir, out_md, title, command = argv[1:5]
    rows = kernel_stats(run_dir)
    with open(out_md, "w") as f:
        f.write(f"# {title}\n\nCommand (from /tmp with TMPDIR=/tmp):\n\n    {command}\n\n")
        f.write("| kernel | calls | average (us) | min (us) | max (us) | share |\n|---|---|---|---|---|---|\n")
        for r in rows:
            f.write(f"| {short_name(r['Name'])} | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                    f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                    f"{float(r['Percentage']):.1f}% |\n")
    print(open(out_md).read())


if __name__ == "__main__":
    main(sys.argv)
