"""Where the pass kernel's time goes, phase by phase.

    python3 -m paper_2609_03311_amd._build timers      (on the build host)
    python3 -m paper_2609_03311_amd.phase_timing CONFIG [--steps N]

Runs the full-layer attention of a synthetic workload (the pass kernel,
``kernel_variant`` 8) on libdopr_timers.so, the library built with the pass
kernel's per-phase cycle counters compiled in, and prints a summary: for
each wave of the 8-wave block, the share of its cycles in each phase
(hand-over, prefix staging, pair search, own-chunk loads, q^ prologue,
waits and barriers, prefix and own products, output), the number of units
and passes, and the share of the near-empty passes (at most 32 rows).  The
counters are ``s_memtime`` cycles read by every wave at the phase marks;
the marks themselves cost a few percent, so the step time printed is the
instrumented kernel's, not the product's.
"""
from __future__ import annotations

import argparse
import ctypes
import os
import sys

import numpy as np

import paper_2609_03311_amd as pkg
from paper_2609_03311_amd import _build, profiling

PHASES = ["unit hand-over", "prefix loads issued", "pair search",
          "own loads issued", "q rows + q^ prologue", "wait for loads",
          "barrier before products", "prefix chunks", "own chunks: products",
          "own chunks: barriers", "own chunks: next loads", "epilogue (O, LSE)",
          "barrier at pass end", "next unit claim"]
N_SLOTS = 18  # the kernel's kPtSlots: the phases, then the counts
UNITS, PASSES, TAIL_CYC, TAILS = 14, 15, 16, 17


def run(config: str, steps: int):
    if not os.path.exists(_build.TIMERS_LIB):
        raise SystemExit(f"{_build.TIMERS_LIB} is missing: build it with "
                         "`python3 -m paper_2609_03311_amd._build timers`")
    pkg.LIB_PATH = _build.TIMERS_LIB
    import torch
    import workloads
    from paper_2609_03311_amd import pipeline

    dev = "cuda"
    st = workloads.make(config)
    k_src, v_src, _, _ = workloads.prefix_source(st, dev, 1)
    on = workloads.online_inputs(st, dev, 3)
    prm = workloads.params(st, dev, 6)
    store = pipeline.make_store(st.doc_len, st.n_kv_heads, k_src, v_src,
                                device=dev)
    step = pipeline.OnlineStep(store, n_pairs=st.n_pairs,
                               n_q_heads=st.n_q_heads,
                               total_tokens=st.n_tokens,
                               max_tokens=int(st.seqlens.max()),
                               kernel_variant=8, device=dev)
    ids = torch.from_numpy(st.doc_ids).to(dev)
    cu = torch.from_numpy(st.cu_seqlens).to(dev)

    def once():
        step.attention(0, ids, cu, on["q"], on["k"], on["v"],
                       prm["q_norm_w"], prm["k_norm_w"])

    L = pkg.lib()
    read = L.dopr_pass_phase_read
    read.argtypes = [ctypes.POINTER(ctypes.c_ulonglong), ctypes.c_int]
    read.restype = ctypes.c_int
    buf = (ctypes.c_ulonglong * (8 * N_SLOTS))()
    once()
    torch.cuda.synchronize()
    if read(buf, 1) != 0:
        raise SystemExit("dopr_pass_phase_read failed")
    a = torch.cuda.Event(enable_timing=True)
    b = torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(steps):
        once()
    b.record()
    torch.cuda.synchronize()
    if read(buf, 1) != 0:
        raise SystemExit("dopr_pass_phase_read failed")
    t = np.array(list(buf), dtype=np.float64).reshape(8, N_SLOTS)
    return t, a.elapsed_time(b) / steps


def summary(config: str, steps: int, t, ms: float, command: str) -> str:
    cyc = t[:, :len(PHASES)]
    tot = cyc.sum(axis=1)
    out = ["# Pass-kernel phases (s_memtime cycles per wave, instrumented "
           "build)", f"command: {command}",
           f"kernel_source_sha: {profiling.kernel_source_sha()}",
           f"workload: {config}, {steps} steps, kernel_variant 8",
           f"instrumented step: {ms:.3f} ms (attention + grouping)",
           f"units per step: {t[0, UNITS] / steps:.0f}, passes per step: "
           f"{t[0, PASSES] / steps:.0f} "
           f"({t[0, PASSES] / max(t[0, UNITS], 1):.2f} per unit)",
           f"cycles per pass (wave 0): {tot[0] / max(t[0, PASSES], 1):.0f}",
           f"passes of at most 32 rows: {t[0, TAILS] / steps:.0f} per step, "
           f"{t[0, TAIL_CYC] / max(t[0, TAILS], 1):.0f} cycles each, "
           f"{100 * t[0, TAIL_CYC] / tot[0]:.1f} % of wave 0's cycles", "",
           f"{'phase':<26}" + "".join(f"{'w' + str(w):>8}" for w in range(8))
           + f"{'mean':>8}"]
    share = 100 * cyc / tot[:, None]
    for i, name in enumerate(PHASES):
        out.append(f"{name:<26}" + "".join(f"{share[w, i]:7.2f}%"
                                           for w in range(8))
                   + f"{share[:, i].mean():7.2f}%")
    return "\n".join(out) + "\n"


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("config")
    ap.add_argument("--steps", type=int, default=5)
    args = ap.parse_args(argv)
    t, ms = run(args.config, args.steps)
    command = (f"python3 -m paper_2609_03311_amd.phase_timing {args.config} "
               f"--steps {args.steps} (library: python3 -m "
               "paper_2609_03311_amd._build timers)")
    sys.stdout.write(summary(args.config, args.steps, t, ms, command))


if __name__ == "__main__":
    main()
