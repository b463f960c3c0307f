"""Summaries of rocprofv3 output for the attention kernel (text, a few KB).

    python3 -m paper_2609_03311_amd.profiling stats TRACE_DIR --command CMD
    python3 -m paper_2609_03311_amd.profiling traffic FETCH_DIR WRITE_DIR \
        --command CMD [--kernel REGEX]
    python3 -m paper_2609_03311_amd.profiling pmc RUN_DIR... --command CMD
    python3 -m paper_2609_03311_amd.profiling benchtable JSONL... \
        --command CMD

`stats` condenses `rocprofv3 --kernel-trace --stats` (run_kernel_stats.csv)
into a per-kernel table.  `traffic` turns two `--pmc FETCH_SIZE` /
`--pmc WRITE_SIZE` runs of `bench.py --copy-calibration` into HBM bytes per
launch of the attention kernel: each counter (KiB per dispatch) is scaled by
what the same counter reads for the calibration kernel, a plain streaming
kernel that reads and writes exactly `CALIB_BYTES`.  `pmc` condenses
`--pmc` runs of shader counters into MFMA, VALU and LDS utilisation and wait
fractions per kernel.  Every summary records a hash of the kernels' sources
so a reader can tell whether the figures still describe the code.

The full layer's attention is two launches: `k_own_khat` (k^ of every
online token) and the pass kernel `k_pass_attn`; both are timed and
counted together as one attention step.
"""
import argparse
import csv
import hashlib
import os
import re
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
KERNEL_SOURCES = ("csrc/attn.hip", "csrc/attn_common.hpp", "csrc/stream.hip",
                  "csrc/internal.hpp")
# the sources each kind of summary describes (its hash is recorded with it)
SOURCE_SETS = {
    "attention": KERNEL_SOURCES,
    "salience": ("csrc/salience.hip", "csrc/internal.hpp"),
    "store": ("csrc/store.hip", "csrc/internal.hpp"),
    "layer": ("csrc/layer.hip", "csrc/group.hip", "csrc/score.hip")
    + KERNEL_SOURCES,
}
# the attention launches of each path on the Qwen3-8B-shaped workload (head
# size 128): k^ precompute + pass kernel (full layer); one wave per 32-row
# unit (score rows, every prefix at most 512 slots).  Same at head size 64.
ATTN_KERNEL = r"k_own_khat<128>|k_pass_attn<128>"
SCORE_KERNEL = r"k_score_rows<128>"
ATTN_KERNEL_D64 = r"k_own_khat<64>|k_pass_attn<64>"
SCORE_KERNEL_D64 = r"k_score_rows<64>"
CALIB_KERNEL = r"bitwise_not"
CALIB_BYTES = 1 << 30


def _code_only(text):
    """The source without comments and with whitespace runs collapsed, so
    that an edit to a comment leaves the hash alone."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_sha(kind="attention"):
    """Hash of one kind of kernel's code (comments and layout ignored)."""
    h = hashlib.sha256()
    for rel in SOURCE_SETS[kind]:
        with open(os.path.join(HERE, rel), encoding="utf-8") as f:
            h.update(_code_only(f.read()).encode())
    return h.hexdigest()[:16]


def _sha_lines(kind):
    lines = [f"kernel_source_sha: {kernel_source_sha(kind)}"]
    if kind != "attention":
        lines.append("kernel_sources: " + " ".join(
            os.path.basename(r) for r in SOURCE_SETS[kind]))
    return lines


def short_name(name, width=72):
    n = re.sub(r"\(.*$", "", name.replace("(anonymous namespace)::", ""))
    n = n.replace("void ", "").replace("dopr::", "")
    return n if len(n) <= width else n[:width - 3] + "..."


def _rows(path):
    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def stats(trace_dir, command, top=12, sources="attention"):
    rows = _rows(os.path.join(trace_dir, "run_kernel_stats.csv"))
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    out = ["# rocprofv3 kernel statistics", f"command: {command}",
           *_sha_lines(sources), "",
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
    """Values of one counter, per dispatch, of every kernel matching
    `pattern`: {kernel name: [values]}."""
    vals = {}
    for r in _rows(os.path.join(run_dir, "run_counter_collection.csv")):
        if r["Counter_Name"] == counter and re.search(pattern,
                                                      r["Kernel_Name"]):
            vals.setdefault(short_name(r["Kernel_Name"]), []).append(
                float(r["Counter_Value"]))
    if not vals:
        raise SystemExit(f"no {counter} rows for /{pattern}/ in {run_dir}")
    return vals


def _per_step(vals):
    """Sum over the matched kernels of each one's mean per dispatch (one
    attention step launches each of them once)."""
    return sum(sum(v) / len(v) for v in vals.values())


def traffic(fetch_dir, write_dir, command, kernel=ATTN_KERNEL,
            sources="attention"):
    f_att = _counter(fetch_dir, "FETCH_SIZE", kernel)
    w_att = _counter(write_dir, "WRITE_SIZE", kernel)
    f_cal = [x for v in _counter(fetch_dir, "FETCH_SIZE", CALIB_KERNEL).values()
             for x in v]
    w_cal = [x for v in _counter(write_dir, "WRITE_SIZE", CALIB_KERNEL).values()
             for x in v]
    kib = 1024.0
    f_scale = CALIB_BYTES / (max(f_cal) * kib)
    w_scale = CALIB_BYTES / (max(w_cal) * kib)
    f_avg = _per_step(f_att)
    w_avg = _per_step(w_att)
    read_b = f_avg * kib * f_scale
    write_b = w_avg * kib * w_scale
    out = [
        "# HBM traffic of the attention kernel (rocprofv3 --pmc)",
        f"command: {command}",
        f"kernel: /{kernel}/",
        *_sha_lines(sources),
        "dispatches: " + ", ".join(
            f"{k} fetch {len(f_att[k])} write {len(w_att.get(k, []))}"
            for k in sorted(f_att)),
        *[f"fetch_kib_per_dispatch[{k}]: {sum(v) / len(v):.1f}"
          for k, v in sorted(f_att.items())],
        *[f"write_kib_per_dispatch[{k}]: {sum(v) / len(v):.1f}"
          for k, v in sorted(w_att.items())],
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


# Shader counters summarised by `pmc` (each pass of rocprofv3 --pmc holds
# at most 8 SQ counters and GRBM_GUI_ACTIVE; one pass per group).
PMC_PASSES = (
    "SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 "
    "SQ_INSTS_MFMA SQ_INSTS_VALU SQ_ACTIVE_INST_VALU SQ_INSTS_LDS "
    "SQ_WAVE_CYCLES GRBM_GUI_ACTIVE",
    "SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_WAIT_INST_LDS SQ_ACTIVE_INST_ANY "
    "SQ_ACTIVE_INST_LDS SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE "
    "SQ_ACTIVE_INST_VMEM GRBM_GUI_ACTIVE",
)


def _agent(run_dir):
    for r in _rows(os.path.join(run_dir, "run_agent_info.csv")):
        if r.get("Name", "").startswith("gfx"):
            return r
    raise SystemExit(f"no GPU agent in {run_dir}")


def pmc(run_dirs, command, kernel=ATTN_KERNEL, sources="attention"):
    """Per matched kernel: the mean per dispatch of every counter found in
    the runs, and the utilisations the ROCm derived metrics define.
    GRBM_GUI_ACTIVE is summed over the chip's XCDs in the counter file, so
    the busy-cycle denominators use it divided by the XCD count."""
    ag = _agent(run_dirs[0])
    n_xcc, n_cu = int(ag["Num_Xcc"]), int(ag["Cu_Count"])
    n_simd = int(ag["Simd_Count"])
    per = {}    # kernel -> counter -> [values]
    meta = {}   # kernel -> resources and duration
    for d in run_dirs:
        for r in _rows(os.path.join(d, "run_counter_collection.csv")):
            if not re.search(kernel, r["Kernel_Name"]):
                continue
            k = short_name(r["Kernel_Name"])
            per.setdefault(k, {}).setdefault(r["Counter_Name"], []).append(
                float(r["Counter_Value"]))
            meta.setdefault(k, {
                "arch_vgpr": r["VGPR_Count"], "accum_vgpr": r["Accum_VGPR_Count"],
                "sgpr": r["SGPR_Count"], "lds_bytes": r["LDS_Block_Size"],
                "scratch_bytes_per_lane": r["Scratch_Size"],
                "workgroup": r["Workgroup_Size"], "grid": r["Grid_Size"]})
            meta[k].setdefault("dur", []).append(
                int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    if not per:
        raise SystemExit(f"no counter rows for /{kernel}/ in {run_dirs}")
    what = "attention launches" if sources == "attention" else "launches"
    out = [f"# Shader counters of the {what} (rocprofv3 --pmc)",
           f"command: {command}", f"kernel: /{kernel}/",
           *_sha_lines(sources),
           f"agent: {ag['Name']}, {n_xcc} XCDs, {n_cu} CUs, {n_simd} SIMDs",
           ""]
    tot_busy = tot_cycles = tot_mops = tot_dur = 0.0
    for k in sorted(per):
        c = {n: sum(v) / len(v) for n, v in per[k].items()}
        m = meta[k]
        dur = sum(m["dur"]) / len(m["dur"])
        gui = c.get("GRBM_GUI_ACTIVE", 0.0) / n_xcc   # cycles per XCD
        out.append(f"[{k}]")
        out.append(f"  mean_duration_us: {dur / 1e3:.1f}")
        for key in ("arch_vgpr", "accum_vgpr", "sgpr", "lds_bytes",
                    "scratch_bytes_per_lane", "workgroup", "grid"):
            out.append(f"  {key}: {m[key]}")
        for n in sorted(c):
            out.append(f"  {n}: {c[n]:.6g}")
        if gui > 0:
            busy = c.get("SQ_VALU_MFMA_BUSY_CYCLES", 0.0)
            out.append(f"  mfma_busy_pct: {100 * busy / (gui * n_simd):.2f}")
            out.append("  valu_busy_pct: "
                       f"{100 * c.get('SQ_ACTIVE_INST_VALU', 0.0) / n_cu / gui:.2f}")
            out.append("  lds_util_pct: "
                       f"{100 * c.get('SQ_LDS_IDX_ACTIVE', 0.0) / n_cu / gui:.2f}")
            out.append("  lds_bank_conflict_pct: "
                       f"{100 * c.get('SQ_LDS_BANK_CONFLICT', 0.0) / n_cu / gui:.2f}")
            tot_busy += busy
            tot_cycles += gui * n_simd
        if c.get("SQ_WAVE_CYCLES"):
            w = c["SQ_WAVE_CYCLES"]
            for n in ("SQ_WAIT_ANY", "SQ_WAIT_INST_ANY", "SQ_ACTIVE_INST_ANY"):
                if n in c:
                    out.append(f"  {n.lower()}_frac_of_wave_cycles: "
                               f"{c[n] / w:.3f}")
        if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in c and dur > 0:
            fl = 512 * c["SQ_INSTS_VALU_MFMA_MOPS_BF16"]
            out.append(f"  mfma_bf16_flop: {fl:.6g}")
            out.append(f"  mfma_bf16_tflops: {fl / (dur * 1e-9) / 1e12:.1f}")
            tot_mops += fl
            tot_dur += dur
    if tot_cycles > 0:
        out += ["", f"mfma_busy_frac: {tot_busy / tot_cycles:.4f}"]
    if tot_dur > 0:
        out.append(f"mfma_bf16_tflops: {tot_mops / (tot_dur * 1e-9) / 1e12:.1f}")
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


def bench_table(paths, command):
    """One row per bench.py JSON line (files of JSON lines; other lines are
    skipped): workload, path, queue order, step and attention times, the
    roofline figures, the throughput, and where a committed profile of the
    kernel exists for the current sources, its measured HBM bytes per
    launch and MFMA busy fraction."""
    import json
    out = ["# bench.py on each workload and path (one MI355X)",
           f"command: {command}", "",
           f"{'workload':20s} {'path':34s} {'qo':>2s} {'step ms':>9s} "
           f"{'attn ms':>9s} {'achieved':>16s} {'frac':>6s} "
           f"{'throughput':>22s} {'HBM GB':>8s} {'mfma':>6s}"]
    for path in paths:
        with open(path) as f:
            for line in f:
                line = line.strip()
                if not line.startswith("{"):
                    continue
                try:
                    d = json.loads(line)
                except ValueError:
                    continue
                cfg = d.get("config", {})
                r = d.get("roofline") or {}
                qo = cfg.get("queue_order")
                attn = d.get("attention_ms")
                tr = r.get("traffic")
                mu = d.get("mfma_util")
                label = cfg.get("path") or (
                    "full layer, prefix budget sweep" if "k_infer" in cfg
                    else d.get("metric", "?"))
                out.append(
                    f"{str(cfg.get('name', '?')):20s} "
                    f"{str(label)[:34]:34s} "
                    f"{'' if qo is None else qo:>2} "
                    f"{d.get('ms_per_step', float('nan')):9.3f} "
                    f"{'' if attn is None else f'{attn:9.3f}':>9s} "
                    f"{r.get('achieved', float('nan')):9.1f} "
                    f"{str(r.get('unit', '')):>6s} "
                    f"{r.get('frac', float('nan')):6.4f} "
                    f"{d.get('value', float('nan')):12.1f} "
                    f"{str(d.get('unit', ''))[:9]:>9s} "
                    f"{'' if tr is None else f'{tr / 1e9:8.2f}':>8s} "
                    f"{'' if mu is None else f'{mu:6.3f}':>6s}")
                if "k_infer" in cfg:
                    out.append(f"{'':20s}   K_infer {cfg['k_infer']}: store "
                               f"{d.get('store_gb_per_layer')} GB per layer, "
                               f"{d.get('doc_state_kb_all_layers')} KB per "
                               f"document over 36 layers, "
                               f"{d.get('us_per_pair')} us per pair, "
                               f"algorithmic {d.get('algorithmic_gb')} GB")
                cb = d.get("cpu_baseline")
                if cb:
                    out.append(f"{'':20s}   cpu_baseline {cb.get('value')} "
                               f"{cb.get('unit')} on {cb.get('cores')} "
                               f"threads ({cb.get('kind')})")
    return "\n".join(out) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("trace_dir")
    a.add_argument("--command", required=True)
    a.add_argument("--sources", default="attention", choices=SOURCE_SETS)
    b = sub.add_parser("traffic")
    b.add_argument("fetch_dir")
    b.add_argument("write_dir")
    b.add_argument("--command", required=True)
    b.add_argument("--kernel", default=ATTN_KERNEL)
    b.add_argument("--sources", default="attention", choices=SOURCE_SETS)
    c = sub.add_parser("pmc")
    c.add_argument("run_dirs", nargs="+")
    c.add_argument("--command", required=True)
    c.add_argument("--kernel", default=ATTN_KERNEL)
    c.add_argument("--sources", default="attention", choices=SOURCE_SETS)
    t = sub.add_parser("benchtable")
    t.add_argument("jsonl", nargs="+")
    t.add_argument("--command", required=True)
    args = ap.parse_args(argv)
    if args.cmd == "benchtable":
        sys.stdout.write(bench_table(args.jsonl, args.command))
    elif args.cmd == "stats":
        sys.stdout.write(stats(args.trace_dir, args.command,
                               sources=args.sources))
    elif args.cmd == "pmc":
        sys.stdout.write(pmc(args.run_dirs, args.command, args.kernel,
                             args.sources))
    else:
        sys.stdout.write(traffic(args.fetch_dir, args.write_dir, args.command,
                                 args.kernel, args.sources))


if __name__ == "__main__":
    main()
