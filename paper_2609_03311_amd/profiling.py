"""Summaries of rocprofv3 output for the attention kernel (text, a few KB).

    python3 -m paper_2609_03311_amd.profiling stats TRACE_DIR --command CMD
    python3 -m paper_2609_03311_amd.profiling traffic FETCH_DIR WRITE_DIR \
        --command CMD [--kernel REGEX]

`stats` condenses `rocprofv3 --kernel-trace --stats` (run_kernel_stats.csv)
into a per-kernel table.  `traffic` turns two `--pmc FETCH_SIZE` /
`--pmc WRITE_SIZE` runs of `bench.py --copy-calibration` into HBM bytes per
launch of the attention kernel: each counter (KiB per dispatch) is scaled by
what the same counter reads for the calibration kernel, a plain streaming
kernel that reads and writes exactly `CALIB_BYTES`.  The summary records a
hash of the kernel's sources so a reader can tell whether the figures still
describe the code.
"""
import argparse
import csv
import hashlib
import os
import re
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = ("csrc/attn.hip", "csrc/internal.hpp")
# the dominant kernel of each path on the Qwen3-8B-shaped workload (head
# size 128): 8 waves, 256 slots resident (full layer); two 4-wave blocks per
# CU (score rows).  At head size 64 the same shapes hold 512 and 192 slots.
ATTN_KERNEL = r"k_prefix_attn<8, ?1, ?false, ?false, ?128, ?8>"
SCORE_KERNEL = r"k_prefix_attn<4, ?1, ?false, ?true, ?128, ?3>"
ATTN_KERNEL_D64 = r"k_prefix_attn<8, ?1, ?false, ?false, ?64, ?16>"
SCORE_KERNEL_D64 = r"k_prefix_attn<4, ?1, ?false, ?true, ?64, ?6>"
CALIB_KERNEL = r"bitwise_not"
CALIB_BYTES = 1 << 30


def kernel_source_sha():
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(HERE, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def short_name(name, width=72):
    n = re.sub(r"\(.*$", "", name.replace("(anonymous namespace)::", ""))
    n = n.replace("void ", "").replace("dopr::", "")
    return n if len(n) <= width else n[:width - 3] + "..."


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def stats(trace_dir, command, top=12):
    rows = _rows(os.path.join(trace_dir, "run_kernel_stats.csv"))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = ["# rocprofv3 kernel statistics", f"command: {command}",
           f"kernel_source_sha: {kernel_source_sha()}", "",
           f"{'kernel':<72} {'calls':>6} {'avg_us':>11} {'min_us':>11} "
           f"{'max_us':>11} {'pct':>6}"]
    for r in rows[:top]:
        out.append(f"{short_name(r['Name']):<72} {int(r['Calls']):>6} "
                   f"{float(r['AverageNs']) / 1e3:>11.1f} "
                   f"{float(r['MinNs']) / 1e3:>11.1f} "
                   f"{float(r['MaxNs']) / 1e3:>11.1f} "
                   f"{float(r['Percentage']):>6.2f}")
    return "\n".join(out) + "\n"


def _counter(run_dir, counter, pattern):
    vals = []
    for r in _rows(os.path.join(run_dir, "run_counter_collection.csv")):
        if r["Counter_Name"] == counter and re.search(pattern,
                                                      r["Kernel_Name"]):
            vals.append(float(r["Counter_Value"]))
    if not vals:
        raise SystemExit(f"no {counter} rows for /{pattern}/ in {run_dir}")
    return vals


def traffic(fetch_dir, write_dir, command, kernel=ATTN_KERNEL):
    f_att = _counter(fetch_dir, "FETCH_SIZE", kernel)
    w_att = _counter(write_dir, "WRITE_SIZE", kernel)
    f_cal = _counter(fetch_dir, "FETCH_SIZE", CALIB_KERNEL)
    w_cal = _counter(write_dir, "WRITE_SIZE", CALIB_KERNEL)
    kib = 1024.0
    f_scale = CALIB_BYTES / (max(f_cal) * kib)
    w_scale = CALIB_BYTES / (max(w_cal) * kib)
    f_avg = sum(f_att) / len(f_att)
    w_avg = sum(w_att) / len(w_att)
    read_b = f_avg * kib * f_scale
    write_b = w_avg * kib * w_scale
    out = [
        "# HBM traffic of the attention kernel (rocprofv3 --pmc)",
        f"command: {command}",
        f"kernel: /{kernel}/",
        f"kernel_source_sha: {kernel_source_sha()}",
        f"dispatches: fetch {len(f_att)}, write {len(w_att)}",
        f"fetch_kib_per_dispatch: {f_avg:.1f}",
        f"write_kib_per_dispatch: {w_avg:.1f}",
        f"calibration: /{CALIB_KERNEL}/ reads and writes {CALIB_BYTES} B; "
        f"FETCH_SIZE {max(f_cal):.1f} KiB, WRITE_SIZE {max(w_cal):.1f} KiB",
        f"fetch_scale: {f_scale:.4f}",
        f"write_scale: {w_scale:.4f}",
        f"read_bytes_per_launch: {read_b:.0f}",
        f"write_bytes_per_launch: {write_b:.0f}",
        f"traffic_bytes_per_launch: {read_b + write_b:.0f}",
    ]
    return "\n".join(out) + "\n"


def read_summary(path):
    """key: value lines of a summary written by this module."""
    vals = {}
    if not os.path.exists(path):
        return vals
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith("#"):
                k, v = line.split(":", 1)
                vals[k.strip()] = v.strip()
    return vals


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("trace_dir")
    a.add_argument("--command", required=True)
    b = sub.add_parser("traffic")
    b.add_argument("fetch_dir")
    b.add_argument("write_dir")
    b.add_argument("--command", required=True)
    b.add_argument("--kernel", default=ATTN_KERNEL)
    args = ap.parse_args(argv)
    if args.cmd == "stats":
        sys.stdout.write(stats(args.trace_dir, args.command))
    else:
        sys.stdout.write(traffic(args.fetch_dir, args.write_dir, args.command,
                                 args.kernel))


if __name__ == "__main__":
    main()
