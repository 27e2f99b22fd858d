"""HBM traffic of the scoring kernel from two rocprofv3 counter runs.

    rocprofv3 --pmc FETCH_SIZE --output-format csv -d <dir_fetch> -o run -- python3 bench.py \
        --steps 5 --warmup 2 --no-cpu-baseline --no-configs --no-decode --no-entropy --no-fullspan \
        --copy-calibration
    rocprofv3 --pmc WRITE_SIZE --output-format csv -d <dir_write> -o run -- (same command)
    python -m paper_2606_15157_amd.pmc_summary <dir_fetch> <dir_write> <out.json> <out.md>

    python -m paper_2606_15157_amd.pmc_summary --sq <out.md> <dir> [<dir> ...]

The second form tabulates SQ counters of the scoring kernel from one or more rocprofv3 --pmc
runs (median over the kernel's dispatches in each run): shares of SQ_WAVE_CYCLES and instruction
counts per wave and per pipeline iteration.

FETCH_SIZE / WRITE_SIZE (KiB per dispatch) are scaled by what the same counter reads for the
plain 1 GiB device copy that --copy-calibration runs (bytes known exactly), and the result is
stored with the hash of the kernel source it was measured on.
"""
from __future__ import annotations

import csv
import glob
import hashlib
import json
import os
import statistics
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# the scoring kernel's sources: a traffic record is taken on exactly these texts
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2606_15157_amd", "csrc", n) for n in ("prefill.hip", "lds_dma.h", "rkv_internal.h")]
SCORE_NAME = "score_pipe_kernel<1, false>"
COPY_NAME = "__amd_rocclr_copyBuffer"
COPY_BYTES = 1 << 30
# the profiled program: the headline route only, plus the 1 GiB calibration copy
BENCH_CMD = ("python3 bench.py --steps 5 --warmup 2 --no-cpu-baseline --no-configs --no-decode --no-entropy "
             "--no-fullspan --copy-calibration")


def per_dispatch(run_dir: str, counter: str):
    """{kernel name: [counter value per dispatch]} from a rocprofv3 counter_collection CSV."""
    path = glob.glob(os.path.join(run_dir, "**", "*counter_collection.csv"), recursive=True)
    if not path:
        raise FileNotFoundError(f"no counter_collection.csv under {run_dir}")
    acc = {}
    for row in csv.DictReader(open(path[0])):
        if row["Counter_Name"] != counter:
            continue
        key = (row["Kernel_Name"], row["Dispatch_Id"])
        acc[key] = acc.get(key, 0.0) + float(row["Counter_Value"])   # sum over XCDs / instances
    out = {}
    for (name, _), v in acc.items():
        out.setdefault(name, []).append(v)
    return out


def pick(d, needle):
    for name, vals in d.items():
        if needle in name:
            return name, vals
    raise KeyError(needle)


def kernel_source_hash() -> str:
    """SHA-256 over the scoring kernel's source files (names and contents, in order)."""
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        h.update(os.path.basename(path).encode())
        h.update(open(path, "rb").read())
    return h.hexdigest()


def main(argv):
    fetch_dir, write_dir, out_json, out_md = argv[1:5]
    fetch = per_dispatch(fetch_dir, "FETCH_SIZE")
    write = per_dispatch(write_dir, "WRITE_SIZE")
    _, copy_f = pick(fetch, COPY_NAME)
    _, copy_w = pick(write, COPY_NAME)
    cf, cw = max(copy_f), max(copy_w)          # the 1 GiB calibration copy is the largest
    f_scale, w_scale = COPY_BYTES / cf, COPY_BYTES / cw
    name, sf = pick(fetch, SCORE_NAME)
    _, sw = pick(write, SCORE_NAME)
    read_b = statistics.median(sf) * f_scale
    write_b = statistics.median(sw) * w_scale
    rec = {
        "kernel": name,
        "kernel_source_sha256": kernel_source_hash(),
        "fetch_kib_median": statistics.median(sf),
        "write_kib_median": statistics.median(sw),
        "copy_calibration_bytes": COPY_BYTES,
        "copy_fetch_kib": cf,
        "copy_write_kib": cw,
        "fetch_scale": f_scale,
        "write_scale": w_scale,
        "hbm_read_bytes_per_launch": read_b,
        "hbm_write_bytes_per_launch": write_b,
        "hbm_bytes_per_launch": read_b + write_b,
        "dispatches": len(sf),
    }
    json.dump(rec, open(out_json, "w"), indent=1)
    with open(out_md, "w") as f:
        f.write(f"# HBM traffic of {name} (32-layer mixed route, L=8192)\n\n")
        f.write("Commands (each in its own run, from /tmp with TMPDIR=/tmp):\n\n")
        f.write(f"    rocprofv3 --pmc FETCH_SIZE --output-format csv -d <fetch> -o run -- {BENCH_CMD}\n")
        f.write(f"    rocprofv3 --pmc WRITE_SIZE --output-format csv -d <write> -o run -- {BENCH_CMD}\n")
        f.write("    python -m paper_2606_15157_amd.pmc_summary <fetch> <write> <json> <md>\n\n")
        f.write("| quantity | value |\n|---|---|\n")
        for k in ("fetch_kib_median", "write_kib_median", "copy_fetch_kib", "copy_write_kib", "fetch_scale",
                  "write_scale", "hbm_read_bytes_per_launch", "hbm_write_bytes_per_launch", "hbm_bytes_per_launch",
                  "dispatches"):
            f.write(f"| {k} | {rec[k]:.6g} |\n" if isinstance(rec[k], float) else f"| {k} | {rec[k]} |\n")
    print(json.dumps(rec))


SQ_SHARES = ("SQ_WAVE_CYCLES", "SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY", "SQ_ACTIVE_INST_VALU",
             "SQ_ACTIVE_INST_SCA", "SQ_VALU_MFMA_BUSY_CYCLES", "SQ_ACTIVE_INST_LDS", "SQ_WAIT_INST_LDS",
             "SQ_ACTIVE_INST_MISC", "SQ_ACTIVE_INST_VMEM", "SQ_LDS_IDX_ACTIVE", "SQ_LDS_BANK_CONFLICT",
             "SQ_LDS_ADDR_CONFLICT", "SQ_BUSY_CYCLES")
SQ_COUNTS = ("SQ_INSTS_VALU", "SQ_INSTS_SALU", "SQ_INSTS_MFMA", "SQ_INSTS_LDS", "SQ_INSTS_VMEM")


def sq_main(out_md, dirs, iterations=64):
    vals = {}
    for d in dirs:
        path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
        counters = {row["Counter_Name"] for row in csv.DictReader(open(path[0]))}
        for c in counters:
            _, v = pick(per_dispatch(d, c), SCORE_NAME)
            vals[c] = statistics.median(v)
    wc, waves = vals["SQ_WAVE_CYCLES"], vals["SQ_WAVES"]
    with open(out_md, "w") as f:
        f.write(f"# SQ counters of {SCORE_NAME} (32-layer mixed route, L=8192)\n\n")
        f.write("Commands (one run per counter set, from /tmp with TMPDIR=/tmp; median over the dispatches "
                "of each run):\n\n")
        for d in dirs:
            path = glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)
            cs = sorted({row["Counter_Name"] for row in csv.DictReader(open(path[0]))})
            f.write(f"    rocprofv3 --pmc {' '.join(cs)} --output-format csv -d <dir> -o run -- {BENCH_CMD}\n")
        f.write(f"    python -m paper_2606_15157_amd.pmc_summary --sq <out.md> <dir> ...\n\n")
        f.write(f"{waves:.0f} waves; each runs {iterations} pipeline iterations.\n\n")
        f.write("| counter | value | share of SQ_WAVE_CYCLES |\n|---|---|---|\n")
        for c in SQ_SHARES:
            if c in vals:
                f.write(f"| {c} | {vals[c]:.4g} | {vals[c] / wc:.3f} |\n")
        f.write("\n| instructions | per wave | per wave and iteration |\n|---|---|---|\n")
        for c in SQ_COUNTS:
            if c in vals:
                f.write(f"| {c} | {vals[c] / waves:.0f} | {vals[c] / waves / iterations:.0f} |\n")
    print(open(out_md).read())


if __name__ == "__main__":
    if len(sys.argv) > 1 and sys.argv[1] == "--sq":
        sq_main(sys.argv[2], sys.argv[3:])
    else:
        main(sys.argv)
