#!/usr/bin/env python3
"""Throughput of the DoPR online scoring step on one MI355X.

One step = one batch of (query, document) pairs through one decoder layer's
online path: device-side grouping by document, prefix attention over the HBM
prefix store plus causal own keys (QK-RMSNorm + RoPE, GQA, online softmax),
and the yes/no score head on each pair's score token.  Inputs are seeded
synthetic tensors already resident in HBM when timing starts.

Prints one JSON line: pairs/s per decoder layer (whole job), the attention
kernel's achieved algorithmic HBM GB/s against the 8 TB/s peak, and the
float64 CPU oracle timed on a bounded sample of the same workload.

--path score measures last-layer scoring instead: only each pair's score
token is attended (still over its whole prefix and all its own keys) and
the score head is fused into the attention epilogue.  --path layer measures
one whole decoder layer over the online tokens (projections, norms, SwiGLU
MLP and the prefix attention), MFMA-bound.  --path salience measures the
offline side: salience selection of the prefix slots of a batch of whole
documents (head-averaged attention, column top-p means, top-K), with
--config one of the *_docs batches.  --path ingest times filling the
workload's prefix store (dopr_store_put) and repacking it to the documents
the batch references (dopr_store_copy_docs).  --sweep-kinfer K1,K2,... times the
full path on the same pairs at several inference prefix budgets (every
document holds K slots) and prints one JSON line per budget.
"""
import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("query-doc pairs/sec per decoder layer; achieved HBM GB/s vs "
          "MI355X peak")
METRIC_LAYER = ("query-doc pairs/sec per full decoder layer (projections, "
                "prefix attention, SwiGLU MLP); achieved MFMA TFLOP/s vs "
                "MI355X bf16 dense peak")
METRIC_SCORE = ("query-doc pairs/sec for the last decoder layer (score-token "
                "rows + fused score head); achieved HBM GB/s vs MI355X peak")
METRIC_SALIENCE = ("documents/sec of offline salience selection (head-averaged "
                   "causal attention, column top-p means, top-K); achieved "
                   "MFMA TFLOP/s vs MI355X bf16 dense peak")
PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0

DESCRIPTIONS = {
    "tiny": "tiny: 1 layer, 16q/8kv heads, D=128, 8 docs x 16 slots, "
            "4 queries x (15+1) tokens x 8 docs = 32 pairs",
    "qwen3_0p6b": "Qwen3-0.6B-shaped layer: 16q/8kv heads, D=128, 10k docs x "
                  "32 slots, 64 queries x 100 docs, T=31+1",
    "qwen3_4b": "Qwen3-4B-shaped layer: 32q/8kv heads, D=128, 100k docs x 64 "
                "slots, 4096 pairs Zipf(1.1) reuse, T=8..64+1",
    "qwen3_8b": "Qwen3-8B-shaped layer: 32q/8kv heads, D=128, 20k docs x 256 "
                "slots (2048-token docs at 8x), 256 queries x 100 docs, "
                "T=128+1",
    "qwen3_8b_ragged": "Qwen3-8B-shaped layer, ragged: 32q/8kv heads, "
                       "prefixes 8..256 slots over 1M doc ids, 16384 pairs "
                       "(50% Zipf reuse), T=16..128+1",
    "qwen3_8b_ragged_x8": "as qwen3_8b_ragged with 8x longer (uncompressed) "
                          "prefixes, 64..2048 slots",
    "llama3_8b": "Llama-3-8B-shaped attention (no QK-norm, rope_theta 5e5 "
                 "with Llama-3 frequency rescaling): 32q/8kv heads, D=128, "
                 "the qwen3_8b pairs (20k docs x 256 slots, 256 queries x "
                 "100 docs, T=128+1)",
    "llama3_2_1b": "Llama-3.2-1B-shaped attention (no QK-norm, rope_theta "
                   "5e5 with Llama-3 frequency rescaling): 32q/8kv heads, "
                   "D=64, the qwen3_8b pairs (20k docs x 256 slots, 256 "
                   "queries x 100 docs, T=128+1)",
}
# attention families: QK-norm on (Qwen3) or off with given frequencies
LLAMA_ROPE_THETA = 500000.0


def llama3_rope_inv_freq(head_dim=128, theta=LLAMA_ROPE_THETA, factor=32.0,
                         low_freq_factor=1.0, high_freq_factor=4.0,
                         original_max_position=8192):
    """Rotation frequencies of the Llama-3 family: theta^(-2i/D), with
    wavelengths longer than original_max_position / low_freq_factor slowed
    down by `factor`, those shorter than original_max_position /
    high_freq_factor kept, and a linear blend (in original_max_position /
    wavelength) in between.  float32 [D/2], as the models compute them."""
    inv = theta ** (-np.arange(0, head_dim, 2, dtype=np.float64) / head_dim)
    inv = inv.astype(np.float32).astype(np.float64)
    wavelen = 2.0 * np.pi / inv
    blend = ((original_max_position / wavelen - low_freq_factor) /
             (high_freq_factor - low_freq_factor))
    mid = (1.0 - blend) * inv / factor + blend * inv
    out = np.where(wavelen > original_max_position / low_freq_factor,
                   inv / factor, inv)
    in_band = ((wavelen >= original_max_position / high_freq_factor) &
               (wavelen <= original_max_position / low_freq_factor))
    return np.where(in_band, mid, out).astype(np.float32)


def family_args(config, dev, head_dim=128):
    """(gains_enabled, extra keyword arguments of the attention calls)."""
    if not config.startswith("llama"):
        return True, {}
    import torch
    inv = torch.from_numpy(llama3_rope_inv_freq(head_dim)).to(dev)
    return False, {"rope_theta": LLAMA_ROPE_THETA, "rope_inv_freq": inv}
SALIENCE_DESCRIPTIONS = {
    "qwen3_0p6b_docs": "salience selection, Qwen3-0.6B-shaped final layer: "
                       "16q/8kv heads, D=128, 512 documents x 256 tokens, "
                       "p=8, K=32 slots kept per document",
    "qwen3_4b_docs": "salience selection, Qwen3-4B-shaped final layer: "
                     "32q/8kv heads, D=128, 256 documents x 512 tokens, p=8, "
                     "K=64 slots kept per document",
    "qwen3_8b_docs": "salience selection, Qwen3-8B-shaped final layer: "
                     "32q/8kv heads, D=128, 64 documents x 2048 tokens, p=8, "
                     "K=256 slots kept per document",
}


def log(msg):
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr,
          flush=True)


class HipEvents:
    """Raw hipEvent_t handles (the library records them on its stream)."""

    def __init__(self, n):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.c_void_p]
        self.hip.hipEventElapsedTime.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.ev = []
        for _ in range(n):
            e = ctypes.c_void_p(0)
            rc = self.hip.hipEventCreate(ctypes.byref(e))
            if rc != 0:
                raise RuntimeError(f"hipEventCreate failed: {rc}")
            self.ev.append(e.value)

    def elapsed_ms(self, a, b):
        self.hip.hipEventSynchronize(ctypes.c_void_p(self.ev[b]))
        ms = ctypes.c_float(0)
        rc = self.hip.hipEventElapsedTime(ctypes.byref(ms),
                                          ctypes.c_void_p(self.ev[a]),
                                          ctypes.c_void_p(self.ev[b]))
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed: {rc}")
        return ms.value

    def close(self):
        for e in self.ev:
            self.hip.hipEventDestroy(ctypes.c_void_p(e))


def algorithmic_work(st):
    """Bytes the step must move (each unique prefix once, each online row
    once) and the attention flops."""
    uniq = np.unique(st.doc_ids)
    L = st.doc_len[uniq].astype(np.int64)
    hkv, hq, D = st.n_kv_heads, st.n_q_heads, st.head_dim
    prefix = int(L.sum()) * hkv * D * 2 * 2
    ntok = st.n_tokens
    qkv = ntok * (hq + 2 * hkv) * D * 2
    out = ntok * hq * D * 2
    meta = st.n_pairs * 8 + len(uniq) * 12
    T = st.seqlens.astype(np.int64)
    Lp = st.doc_len[st.doc_ids].astype(np.int64)
    keys = (T * Lp + T * (T + 1) // 2).sum()      # sum_p sum_j (L + j + 1)
    flops = int(4 * hq * D * keys)
    score_bytes = st.n_pairs * hq * D * 2
    return dict(prefix=prefix, qkv=qkv, out=out, meta=meta,
                total=prefix + qkv + out + meta, flops=flops,
                exps=int(hq * keys), unique_docs=int(len(uniq)),
                score_bytes=score_bytes)


def algorithmic_work_score(st, rows):
    """Last-layer scoring: each unique prefix once, every own key and value
    once, the score token's q row, its output row when written (`rows`),
    the head's partial sums (written, read back), the head weights and the
    logits/score; flops of the score rows only."""
    uniq = np.unique(st.doc_ids)
    L = st.doc_len[uniq].astype(np.int64)
    hkv, hq, D = st.n_kv_heads, st.n_q_heads, st.head_dim
    P = st.n_pairs
    prefix = int(L.sum()) * hkv * D * 2 * 2
    kv = st.n_tokens * 2 * hkv * D * 2
    q = P * hq * D * 2
    out = P * hq * D * 2 + P * hq * 4 if rows else 0
    head = P * hq * 3 * 4 * 2 + 3 * hq * D * 2 + P * 12
    meta = P * 8 + len(uniq) * 12
    T = st.seqlens.astype(np.int64)
    Lp = st.doc_len[st.doc_ids].astype(np.int64)
    flops = int(4 * hq * D * (Lp + T).sum())
    return dict(prefix=prefix, qkv=kv + q, out=out + head, meta=meta,
                total=prefix + kv + q + out + head + meta, flops=flops,
                unique_docs=int(len(uniq)))


def layer_work(st, hidden, inter):
    """Flops of one decoder layer over the online tokens: the projections
    (q, k, v, o, gate, up, down) and the attention products."""
    hq, hkv, D = st.n_q_heads, st.n_kv_heads, st.head_dim
    n = st.n_tokens
    proj = 2 * n * hidden * (hq + 2 * hkv) * D + 2 * n * hq * D * hidden
    mlp = 2 * n * hidden * inter * 3
    att = algorithmic_work(st)["flops"]
    return dict(proj=proj, mlp=mlp, attention=att, total=proj + mlp + att)


# The decoder layer's elementwise bound: |y - y_ref| <= atol + rtol |y_ref|
# (about six bf16 roundings feed an output element; the output is bf16).
LAYER_ATOL, LAYER_RTOL = 2e-2, 2.0 ** -7


def cpu_baseline_layer(st, k_src, v_src, doc_off, x, wts, prm, seconds,
                       y=None):
    """The float64 layer oracle on a bounded sample of pairs; with y (the
    GPU layer's output), its rows of the sampled pairs are compared."""
    import torch

    import oracle
    L = oracle.lib()
    threads = oracle.max_threads(L)
    rng = np.random.default_rng(99)
    order = rng.permutation(st.n_pairs)
    cu = st.cu_seqlens.astype(np.int64)
    dev = k_src.device
    wb = {k: bits(v) for k, v in wts.items()}

    def run(pairs):
        docs = np.unique(st.doc_ids[pairs])
        sub_off = np.full(st.n_docs, -1, np.int64)
        idx, pos = [], 0
        for d in docs:
            n = int(st.doc_len[d])
            sub_off[d] = pos
            idx.append(np.arange(doc_off[d], doc_off[d] + n))
            pos += n
        it = torch.from_numpy(np.concatenate(idx)).to(dev)
        tok = np.concatenate([np.arange(cu[p], cu[p + 1]) for p in pairs])
        tt = torch.from_numpy(tok).to(dev)
        lens = cu[pairs + 1] - cu[pairs]
        scu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        xs = bits(x.index_select(0, tt))
        pk, pv = bits(k_src.index_select(0, it)), bits(v_src.index_select(0, it))
        t0 = time.perf_counter()
        yr, _, _ = oracle.decoder_layer(xs, st.doc_ids[pairs], scu,
                                        st.doc_len, sub_off, pk, pv, wb,
                                        bits(prm["q_norm_w"]),
                                        bits(prm["k_norm_w"]),
                                        n_q_heads=st.n_q_heads,
                                        n_kv_heads=st.n_kv_heads, L=L)
        dt = time.perf_counter() - t0
        if y is not None:
            g = y.index_select(0, tt).double().cpu().numpy()
            d = np.abs(g - yr)
            par["max_abs_y"] = max(par["max_abs_y"], float(d.max()))
            par["max_bound_ratio"] = max(
                par["max_bound_ratio"],
                float((d / (LAYER_ATOL + LAYER_RTOL * np.abs(yr))).max()))
            par["pairs"] += len(pairs)
            par["rows"] += int(yr.shape[0])
        return dt

    par = {"max_abs_y": 0.0, "max_bound_ratio": 0.0, "pairs": 0, "rows": 0}
    total_t, total_n, i = 0.0, 0, 0
    while total_t < seconds and i < st.n_pairs:
        n = min(max(1, total_n), st.n_pairs - i)   # doubling batches
        total_t += run(order[i:i + n])
        total_n += n
        i += n
    model, n_aff = host_cpu()
    res = {"value": round(total_n / total_t, 3), "unit": "pairs/s",
           "cores": int(min(threads, n_aff)), "kind": "oracle",
           "sample": f"{total_n} of {st.n_pairs} pairs (seeded random "
                     f"order), float64 decoder-layer oracle (numpy "
                     f"projections, C attention), {total_t:.1f}s",
           "cpu_model": model, "affinity_cpus": n_aff,
           "omp_threads": int(threads)}
    if y is not None:
        for k in ("max_abs_y", "max_bound_ratio"):
            par[k] = float(f"{par[k]:.3e}")
        par["bound"] = f"|dy| <= {LAYER_ATOL} + 2^-7 |y|"
        res["parity"] = par
    return res


def _profile_value(config, variant, path_kind, what, key):
    """A figure of the committed rocprofv3 summary of this workload's
    attention (what: "traffic" or "pmc"), or None when there is none, the
    run used a non-default kernel, or the kernels' sources changed since the
    counters were taken."""
    from paper_2609_03311_amd import profiling
    tag = "k_score_rows" if path_kind == "score" else "k_pass_attn"
    path = os.path.join(ROOT, "profiles", f"{tag}_{config}_{what}.txt")
    vals = profiling.read_summary(path)
    if variant != 0 or key not in vals:
        return None
    if vals.get("kernel_source_sha") != profiling.kernel_source_sha():
        log(f"{os.path.basename(path)} describes other kernel sources; "
            f"{key} = null")
        return None
    return float(vals[key])


def measured_traffic(config, variant, path_kind="full"):
    """HBM bytes (FETCH_SIZE + WRITE_SIZE, calibrated) per attention step."""
    v = _profile_value(config, variant, path_kind, "traffic",
                       "traffic_bytes_per_launch")
    return None if v is None else int(v)


def measured_mfma_util(config, variant, path_kind="full"):
    """Fraction of the SIMDs' cycles their MFMA units were busy during the
    attention launches (SQ_VALU_MFMA_BUSY_CYCLES over SIMDs x active
    cycles), from the committed counter summary."""
    return _profile_value(config, variant, path_kind, "pmc", "mfma_busy_frac")


def bits(t):
    import torch
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(
        np.uint16)


PARITY_TOL = 2e-2   # max-abs on O, lse and s (bf16 inputs, fp32 accumulation)


def host_cpu():
    """The host's CPU model and the number of CPUs this process may run on."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return model, len(os.sched_getaffinity(0))


def cpu_baseline(st, k_src, v_src, doc_off, online, prm, seconds,
                 last_only=False, family=None, got=None):
    """The float64 oracle on a bounded sample of the same workload's pairs
    (deterministic order), on this host's cores.  last_only: the oracle of
    last-layer scoring (score-token rows only).  got: the GPU step's
    outputs (out, lse or None, score), compared with the oracle on every
    sampled pair; the maximum absolute differences go to result["parity"]."""
    import torch

    import oracle
    L = oracle.lib()
    threads = oracle.max_threads(L)
    par = {"max_abs_O": 0.0, "max_abs_lse": None, "max_abs_s": 0.0,
           "pairs": 0, "rows": 0}
    rng = np.random.default_rng(99)
    order = rng.permutation(st.n_pairs)
    cu = st.cu_seqlens.astype(np.int64)
    dev = k_src.device

    def run(pairs):
        docs = np.unique(st.doc_ids[pairs])
        sub_off = np.full(st.n_docs, -1, np.int64)
        idx, pos = [], 0
        for d in docs:
            n = int(st.doc_len[d])
            sub_off[d] = pos
            idx.append(np.arange(doc_off[d], doc_off[d] + n))
            pos += n
        it = torch.from_numpy(np.concatenate(idx)).to(dev)
        tok = np.concatenate([np.arange(cu[p], cu[p + 1]) for p in pairs])
        tt = torch.from_numpy(tok).to(dev)
        lens = cu[pairs + 1] - cu[pairs]
        scu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        args = (st.doc_ids[pairs], scu, st.doc_len, sub_off,
                bits(k_src.index_select(0, it)),
                bits(v_src.index_select(0, it)),
                bits(online["q"].index_select(0, tt)),
                bits(online["k"].index_select(0, tt)),
                bits(online["v"].index_select(0, tt)),
                None if prm["q_norm_w"] is None else bits(prm["q_norm_w"]),
                None if prm["k_norm_w"] is None else bits(prm["k_norm_w"]))
        nw, wh = bits(prm["norm_w"]), bits(prm["w_head"])
        fam = {}
        if family:
            fam = {"rope_theta": family["rope_theta"],
                   "rope_inv_freq": family["rope_inv_freq"].double().cpu()
                   .numpy()}
        t0 = time.perf_counter()
        out, lse, _ = oracle.prefix_attn(*args, n_q_heads=st.n_q_heads,
                                         n_kv_heads=st.n_kv_heads,
                                         last_only=last_only, L=L, **fam)
        h = (out if last_only else out[scu[1:] - 1]).reshape(len(pairs), -1)
        _, s = oracle.score(h, nw, wh, L=L)
        dt = time.perf_counter() - t0
        if got is not None:
            pt = torch.from_numpy(pairs.astype(np.int64)).to(dev)
            rows = pt if last_only else tt
            if got.get("out") is not None:
                g_out = got["out"].index_select(0, rows).double().cpu().numpy()
                par["max_abs_O"] = max(par["max_abs_O"],
                                       float(np.abs(g_out - out).max()))
            if got.get("lse") is not None:
                g_lse = got["lse"].index_select(0, rows).double().cpu().numpy()
                fin = np.isfinite(lse)
                e = float(np.abs(g_lse[fin] - lse[fin]).max()) if fin.any() \
                    else 0.0
                par["max_abs_lse"] = max(par["max_abs_lse"] or 0.0, e)
            g_s = got["score"].index_select(0, pt).double().cpu().numpy()
            par["max_abs_s"] = max(par["max_abs_s"],
                                   float(np.abs(g_s - s).max()))
            par["pairs"] += len(pairs)
            par["rows"] += int(out.shape[0] * out.shape[1])
        return dt

    # calibrate on one pair per thread, then size the sample to the budget
    first = order[:min(threads, st.n_pairs)]
    t_first = run(first)
    per_pair = t_first / len(first) * min(threads, len(first)) / threads
    n_more = int(max(0.0, seconds - t_first) / max(per_pair, 1e-9))
    n_more = min(n_more, st.n_pairs - len(first))
    n_more = n_more // threads * threads
    total_t, total_n = t_first, len(first)
    if n_more > 0:
        more = order[len(first):len(first) + n_more]
        total_t += run(more)
        total_n += len(more)
    model, n_aff = host_cpu()
    res = {"value": round(total_n / total_t, 3), "unit": "pairs/s",
           "cores": int(min(threads, n_aff)), "kind": "oracle",
           "sample": f"{total_n} of {st.n_pairs} pairs (seeded random "
                     f"order), float64 C oracle"
                     f"{' of the score-token rows' if last_only else ''} "
                     f"incl. score head, {total_t:.1f}s",
           "cpu_model": model, "affinity_cpus": n_aff,
           "omp_threads": int(threads)}
    if got is not None:
        for k in ("max_abs_O", "max_abs_lse", "max_abs_s"):
            if par[k] is not None:
                par[k] = float(f"{par[k]:.3e}")
        par["tol"] = PARITY_TOL
        res["parity"] = par
    return res


def salience_work(lens, hq, D=128):
    """Flops of salience selection: the scaled logits of every head over the
    causally visible keys, formed twice (once for each row's log-sum-exp,
    once for the probabilities), and the exponentials of both sweeps."""
    n = np.asarray(lens, np.int64)
    visible = int((n * (n + 1) // 2).sum())
    return dict(flops=2 * 2 * hq * D * visible, exps=2 * hq * visible)


def cpu_baseline_salience(lens, q, k, p, seconds):
    """The float64 salience oracle on a bounded sample of documents."""
    import oracle
    from oracle import salience as sal_oracle
    threads = oracle.max_threads(oracle.lib())
    rng = np.random.default_rng(99)
    order = rng.permutation(len(lens))
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    total_t, n_docs = 0.0, 0
    for d in order:
        t0, t1 = int(cu[d]), int(cu[d + 1])
        qb, kb = bits(q[t0:t1]), bits(k[t0:t1])
        c = time.perf_counter()
        sal_oracle.salience(qb, kb, [0, t1 - t0], 128 ** -0.5, p,
                            n_select=[(t1 - t0) // 8])
        total_t += time.perf_counter() - c
        n_docs += 1
        if total_t >= seconds:
            break
    return {"value": round(n_docs / total_t, 3), "unit": "documents/s",
            "cores": int(threads), "kind": "oracle",
            "sample": f"{n_docs} of {len(lens)} documents (seeded random "
                      f"order), float64 numpy salience oracle incl. top-K, "
                      f"{total_t:.1f}s"}


def bench_salience(args):
    """Offline salience selection of a batch of documents: one step is one
    dopr_salience call (row log-sum-exp, head-averaged attention, column
    top-p means, top-K) over the whole batch, inputs resident in HBM."""
    import torch

    import workloads
    from paper_2609_03311_amd.pipeline import SalienceStep
    lens, hq, hkv = workloads.salience_batch(args.config)
    p = workloads.SALIENCE_TOP_P
    dev = "cuda"
    q, k = workloads.salience_inputs(lens, hq, hkv, dev)
    step = SalienceStep(lens, n_q_heads=hq, n_kv_heads=hkv, top_p=p,
                        ratio=workloads.SALIENCE_RATIO, device=dev)
    torch.cuda.synchronize()
    log(f"{args.config}: {len(lens)} documents x {int(lens[0])} tokens, "
        f"{hq}q/{hkv}kv heads; warming up")
    for _ in range(args.warmup):
        step.run(q, k)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True),
           torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for a, b in ev:
        a.record()
        step.run(q, k)
        b.record()
    t1.record()
    torch.cuda.synchronize()
    if int(step.status.item()) != 0:
        raise SystemExit(f"device status {int(step.status.item())}")
    ms_step = t0.elapsed_time(t1) / args.steps
    call_ms = float(np.mean([a.elapsed_time(b) for a, b in ev]))
    log(f"step {ms_step:.3f} ms, call avg {call_ms:.3f} ms")
    w = salience_work(lens, hq)
    achieved = w["flops"] / (call_ms * 1e-3) / 1e12
    result = {
        "metric": METRIC_SALIENCE,
        "value": round(len(lens) / (ms_step * 1e-3), 1),
        "unit": "documents/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded N(0,1) bf16 final-layer queries and "
                "keys; no datasets or weights)",
        "config": {"workload": SALIENCE_DESCRIPTIONS[args.config],
                   "name": args.config, "documents": int(len(lens)),
                   "tokens": int(lens.sum()), "top_p": p,
                   "path": "offline salience selection",
                   "parallelism": "single GPU"},
        "salience_ms": round(call_ms, 4),
        "exps": w["exps"],
        "roofline": {"bound": "mfma", "achieved": round(achieved, 1),
                     "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": None,
                     "scope": "the whole dopr_salience call (four kernels)"},
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        result["cpu_baseline"] = cpu_baseline_salience(lens, q, k, p,
                                                       args.cpu_seconds)
    print(json.dumps(result), flush=True)


def bench_ingest(args):
    """Store ingest at scale: dopr_store_put of every resident document of
    the workload's store (the offline fill, Sec. 3.3), then a repack with
    dopr_store_copy_docs into a store that keeps only the documents the
    batch references.  Both are streaming copies: HBM-bound; one JSON line
    each."""
    import torch

    import workloads
    from paper_2609_03311_amd import (dopr_check_status, dopr_store_copy_docs,
                                      dopr_store_create, dopr_store_put)
    st = workloads.make(args.config)
    dev = "cuda"
    k_src, v_src, _, cu = workloads.prefix_source(st, dev, 1)
    res = st.resident_docs().astype(np.int32)
    ids = torch.from_numpy(res).to(dev)
    cu_t = torch.from_numpy(cu.astype(np.int64)).to(dev)
    store = dopr_store_create(1, st.n_kv_heads, st.head_dim, st.doc_len)
    kept = np.full(st.n_docs, -1, np.int32)
    used = np.unique(st.doc_ids)
    kept[used] = st.doc_len[used]
    packed = dopr_store_create(1, st.n_kv_heads, st.head_dim, kept)

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        ev = [(torch.cuda.Event(enable_timing=True),
               torch.cuda.Event(enable_timing=True))
              for _ in range(args.steps)]
        for a, b in ev:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        return float(np.mean([a.elapsed_time(b) for a, b in ev]))

    def block_bytes(lens):
        lens = lens.astype(np.int64)
        return int(((lens + (lens + 7) // 8 * 8) * st.n_kv_heads *
                    st.head_dim * 2).sum())

    put_ms = timed(lambda: dopr_store_put(store, 0, ids, cu_t, k_src, v_src))
    copy_ms = timed(lambda: dopr_store_copy_docs(packed, store))
    assert dopr_check_status(store) == 0 and dopr_check_status(packed) == 0
    lens = st.doc_len[res]
    src_bytes = int(lens.astype(np.int64).sum()) * st.n_kv_heads * \
        st.head_dim * 2 * 2
    put_bytes = src_bytes + block_bytes(lens)
    copy_bytes = 2 * block_bytes(st.doc_len[used])
    for kind, ms, nbytes, ndocs, what in (
            ("put", put_ms, put_bytes, len(res),
             "dopr_store_put of every resident document (read canonical "
             "[slots, Hkv, D] states, write K rows and transposed V)"),
            ("repack", copy_ms, copy_bytes, len(used),
             "dopr_store_copy_docs into a store keeping only the documents "
             "the batch references")):
        gbs = nbytes / (ms * 1e-3) / 1e9
        print(json.dumps({
            "metric": "prefix-store ingest: documents/s; achieved HBM GB/s "
                      "vs MI355X peak",
            "value": round(ndocs / (ms * 1e-3), 1), "unit": "documents/s",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": round(ms, 4), "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic",
            "config": {"workload": DESCRIPTIONS[args.config] + "; " + what,
                       "name": f"{args.config}_{kind}", "documents": ndocs,
                       "parallelism": "single GPU"},
            "bytes_moved_gb": round(nbytes / 1e9, 3),
            "roofline": {"bound": "hbm", "achieved": round(gbs, 1),
                         "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(gbs / PEAK_HBM_GBS, 4),
                         "traffic": None}}), flush=True)
        log(f"{kind}: {ms:.3f} ms, {nbytes / 1e9:.2f} GB, {gbs:.0f} GB/s")


def bench_kinfer(args):
    """Same pairs, several inference prefix budgets K_infer (Sec. 4.5, the
    memory and latency axes of the budget trade-off): the store holds K
    slots per document; one JSON line per budget."""
    import torch

    import workloads
    from paper_2609_03311_amd import dopr_check_status, pipeline
    budgets = [int(k) for k in args.sweep_kinfer.split(",") if k]
    base = workloads.make(args.config)
    dev = "cuda"
    online = workloads.online_inputs(base, dev, 3)
    prm = workloads.params(base, dev, 6)
    doc_ids = torch.from_numpy(base.doc_ids).to(dev)
    cu = torch.from_numpy(base.cu_seqlens).to(dev)
    n_layers_model = {1024: 28, 2560: 36, 4096: 36}.get(base.hidden, 1)
    for K in budgets:
        st = workloads.with_prefix_budget(base, K)
        k_src, v_src, _, _ = workloads.prefix_source(st, dev, 1)
        store = pipeline.make_store(st.doc_len, st.n_kv_heads, k_src, v_src,
                                    device=dev)
        del k_src, v_src
        step = pipeline.OnlineStep(store, n_pairs=st.n_pairs,
                                   n_q_heads=st.n_q_heads,
                                   total_tokens=st.n_tokens,
                                   max_tokens=int(st.seqlens.max()),
                                   kernel_variant=args.variant, device=dev)
        ev = HipEvents(2 * args.steps)
        for _ in range(args.warmup):
            step.attention(0, doc_ids, cu, online["q"], online["k"],
                           online["v"], prm["q_norm_w"], prm["k_norm_w"])
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for i in range(args.steps):
            step.attention(0, doc_ids, cu, online["q"], online["k"],
                           online["v"], prm["q_norm_w"], prm["k_norm_w"],
                           timing=(ev.ev[2 * i], ev.ev[2 * i + 1]))
            step.score_head(cu, prm["norm_w"], prm["w_head"])
        t1.record()
        torch.cuda.synchronize()
        ms_step = t0.elapsed_time(t1) / args.steps
        attn = float(np.mean([ev.elapsed_ms(2 * i, 2 * i + 1)
                              for i in range(args.steps)]))
        ev.close()
        if dopr_check_status(store) != 0:
            raise SystemExit(f"device status error at K={K}")
        w = algorithmic_work(st)
        per_doc = K * st.n_kv_heads * st.head_dim * 2 * 2
        achieved = w["total"] / (attn * 1e-3) / 1e9
        res = {
            "metric": METRIC, "value": round(st.n_pairs / (ms_step * 1e-3), 1),
            "unit": "pairs/s", "n_gpus": 1, "steps": args.steps,
            "warmup": args.warmup, "ms_per_step": round(ms_step, 4),
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
            "dtype": "bf16", "data": "synthetic",
            "config": {"workload": DESCRIPTIONS[args.config] +
                       f"; inference prefix budget K_infer={K} slots",
                       "name": f"{args.config}_k{K}", "k_infer": K,
                       "parallelism": "single GPU"},
            "attention_ms": round(attn, 4),
            "us_per_pair": round(ms_step * 1e3 / st.n_pairs, 4),
            "store_gb_per_layer": round(per_doc * int((st.doc_len > 0).sum())
                                        / 1e9, 3),
            "doc_state_kb_all_layers": round(per_doc * n_layers_model / 1024,
                                             1),
            "algorithmic_gb": round(w["total"] / 1e9, 4),
            "prefix_gb": round(w["prefix"] / 1e9, 4),
            "attention_tflops": round(w["flops"] / (attn * 1e-3) / 1e12, 1),
            "roofline": {"bound": "hbm", "achieved": round(achieved, 1),
                         "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": round(achieved / PEAK_HBM_GBS, 4),
                         "traffic": None},
        }
        print(json.dumps(res), flush=True)
        log(f"K_infer={K}: attention {attn:.3f} ms, step {ms_step:.3f} ms, "
            f"{achieved:.0f} GB/s")
        del step, store
        torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="qwen3_8b",
                    choices=sorted(DESCRIPTIONS) +
                    sorted(SALIENCE_DESCRIPTIONS))
    ap.add_argument("--variant", type=int, default=0)
    ap.add_argument("--queue-order", type=int, choices=[0, 1, 2], default=0,
                    help="work-queue order: 0 automatic, 1 natural, "
                         "2 longest-first")
    ap.add_argument("--path", choices=["full", "score", "layer", "salience",
                                       "ingest"],
                    default="full",
                    help="full: every online row of one layer's attention "
                         "(default); score: last-layer scoring (score-token "
                         "rows, fused score head); layer: one whole decoder "
                         "layer; salience: offline salience selection of "
                         "a batch of documents (--config *_docs)")
    ap.add_argument("--no-score-rows", action="store_true",
                    help="with --path score: do not write the score rows "
                         "(the fused head alone)")
    ap.add_argument("--sweep-kinfer", default="",
                    help="comma-separated inference prefix budgets: time the "
                         "full path on the same pairs at each budget")
    ap.add_argument("--cpu-seconds", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain streaming kernel that reads "
                         "and writes 1 GiB, the reference for scaling HBM "
                         "traffic counters")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the online scoring step has "
              "no inter-GPU part (pairs would be sharded by document, each "
              "GPU serving its own shard of the prefix store). Run with "
              "--gpus 1.", file=sys.stderr)
        sys.exit(2)

    if (args.path == "salience") != (args.config in SALIENCE_DESCRIPTIONS):
        ap.error("--path salience goes with a *_docs --config, and a *_docs "
                 "config with --path salience")
    if args.path == "salience":
        bench_salience(args)
        return
    if args.sweep_kinfer:
        bench_kinfer(args)
        return
    if args.path == "ingest":
        bench_ingest(args)
        return

    import torch

    import workloads
    from paper_2609_03311_amd import dopr_check_status, pipeline

    st = workloads.make(args.config)
    dev = "cuda"
    norm_on, fam = family_args(args.config, dev, st.head_dim)
    if not norm_on and args.path == "layer":
        ap.error("--path layer builds the Qwen3 decoder layer (QK-norm on)")
    log(f"{args.config}: P={st.n_pairs} Ntok={st.n_tokens} "
        f"unique docs={len(np.unique(st.doc_ids))}")
    k_src, v_src, doc_off, _ = workloads.prefix_source(st, dev, 1)
    layer_path = args.path == "layer"
    online = None if layer_path else workloads.online_inputs(st, dev, 3)
    prm = workloads.params(st, dev, 6)
    if not norm_on:
        prm["q_norm_w"] = prm["k_norm_w"] = None
    store = pipeline.make_store(st.doc_len, st.n_kv_heads, k_src, v_src,
                                device=dev)
    score_path = args.path == "score"
    if layer_path:
        hidden, inter = workloads.layer_dims(st)
        x = workloads.hidden_states(st, hidden, dev, 11)
        wts = workloads.layer_weights(st, hidden, inter, dev, 21)
        step = pipeline.LayerStep(store, wts, n_pairs=st.n_pairs,
                                  n_q_heads=st.n_q_heads,
                                  total_tokens=st.n_tokens,
                                  max_tokens=int(st.seqlens.max()),
                                  hidden=hidden, intermediate=inter,
                                  kernel_variant=args.variant, device=dev)
        log(f"layer W={hidden} I={inter}: workspace "
            f"{step.workspace.numel() / 2**30:.1f} GiB")
    elif score_path:
        step = pipeline.ScoreStep(store, n_pairs=st.n_pairs,
                                  n_q_heads=st.n_q_heads,
                                  total_tokens=st.n_tokens,
                                  max_tokens=int(st.seqlens.max()),
                                  kernel_variant=args.variant, device=dev,
                                  with_rows=not args.no_score_rows,
                                  queue_order=args.queue_order)
    else:
        step = pipeline.OnlineStep(store, n_pairs=st.n_pairs,
                                   n_q_heads=st.n_q_heads,
                                   total_tokens=st.n_tokens,
                                   max_tokens=int(st.seqlens.max()),
                                   kernel_variant=args.variant, device=dev,
                                   queue_order=args.queue_order)
    doc_ids = torch.from_numpy(st.doc_ids).to(dev)
    cu = torch.from_numpy(st.cu_seqlens).to(dev)
    torch.cuda.synchronize()
    log("inputs resident; warming up")

    if args.copy_calibration:
        # a plain streaming kernel (int32 bitwise NOT) that reads and writes
        # exactly 1 GiB: the scale for the HBM traffic counters
        src = torch.ones(1 << 28, dtype=torch.int32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.bitwise_not(src, out=dst)
        torch.cuda.synchronize()
        log("calibration kernel: 1 GiB read + 1 GiB written")
        del src, dst

    ev = HipEvents(2 * args.steps)

    def one_step(i=None):
        timing = None if i is None else (ev.ev[2 * i], ev.ev[2 * i + 1])
        if layer_path:
            step.run(0, doc_ids, cu, x, prm["q_norm_w"], prm["k_norm_w"],
                     timing=timing)
            return
        if score_path:
            step.run(0, doc_ids, cu, online["q"], online["k"], online["v"],
                     prm["q_norm_w"], prm["k_norm_w"], prm["norm_w"],
                     prm["w_head"], timing=timing, **fam)
            return
        step.attention(0, doc_ids, cu, online["q"], online["k"],
                       online["v"], prm["q_norm_w"], prm["k_norm_w"],
                       timing=timing, **fam)
        step.score_head(cu, prm["norm_w"], prm["w_head"])

    for _ in range(args.warmup):
        one_step()
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t0.record()
    for i in range(args.steps):
        one_step(i)
    t1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_step = t0.elapsed_time(t1) / args.steps
    attn_ms = [ev.elapsed_ms(2 * i, 2 * i + 1) for i in range(args.steps)]
    ev.close()
    status = dopr_check_status(store)
    if status != 0:
        raise SystemExit(f"device status {status} after the timed steps")
    attn_avg = float(np.mean(attn_ms))
    log(f"step {ms_step:.3f} ms (wall {wall / args.steps * 1e3:.3f} ms), "
        f"attention kernel avg {attn_avg:.3f} ms "
        f"(min {min(attn_ms):.3f}, max {max(attn_ms):.3f})")

    if layer_path:
        lw = layer_work(st, hidden, inter)
        w = dict(total=lw["total"], prefix=algorithmic_work(st)["prefix"],
                 flops=lw["attention"],
                 unique_docs=len(np.unique(st.doc_ids)))
        achieved = lw["total"] / (ms_step * 1e-3) / 1e12
        traffic = mfma_util = None
    else:
        w = (algorithmic_work_score(st, not args.no_score_rows) if score_path
             else algorithmic_work(st))
        achieved = w["total"] / (attn_avg * 1e-3) / 1e9
        traffic = measured_traffic(args.config, args.variant, args.path)
        mfma_util = measured_mfma_util(args.config, args.variant, args.path)
    if (score_path and args.no_score_rows) or args.queue_order != 0:
        traffic = None  # the committed profiles were taken without these
        mfma_util = None if args.queue_order != 0 else mfma_util
    result = {
        "metric": (METRIC_LAYER if layer_path else
                   METRIC_SCORE if score_path else METRIC),
        "value": round(st.n_pairs / (ms_step * 1e-3), 1),
        "unit": "pairs/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": ("synthetic (seeded N(0,1) bf16 prefix states, hidden "
                 "states and N(0, 1/fan-in) layer weights; no datasets or "
                 "trained weights)" if layer_path else
                 "synthetic (seeded N(0,1) bf16 prefix states and online "
                 "q/k/v; no datasets or weights)"),
        "config": {
            "workload": DESCRIPTIONS[args.config],
            "name": args.config,
            "pairs": st.n_pairs,
            "online_tokens": st.n_tokens,
            "unique_docs": w["unique_docs"],
            "kernel_variant": args.variant,
            "queue_order": args.queue_order,
            "path": ("decoder layer (hidden %d, intermediate %d)" % (
                hidden, inter) if layer_path else
                     "last-layer scoring" + (", no score rows written"
                                             if args.no_score_rows else "")
                     if score_path else "full online layer"),
            "parallelism": "single GPU",
        },
        "attention_ms": round(attn_avg, 4),
        "algorithmic_gb": round(w["total"] / 1e9, 4),
        "prefix_gb": round(w["prefix"] / 1e9, 4),
        "prefix_gbps": round(w["prefix"] / (attn_avg * 1e-3) / 1e9, 1),
        "attention_tflops": round(w["flops"] / (attn_avg * 1e-3) / 1e12, 1),
        "roofline": ({
            "bound": "mfma",
            "achieved": round(achieved, 1),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
            "traffic": None,
        } if layer_path else {
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": round(achieved / PEAK_HBM_GBS, 4),
            "traffic": traffic,
        }),
        # MFMA busy fraction of the attention launches, from the committed
        # rocprofv3 --pmc summary of the same workload (null without one)
        "mfma_util": mfma_util,
    }
    if layer_path:
        result["algorithmic_gb"] = None   # MFMA-bound: flops, not bytes
        result["layer_tflop"] = round(lw["total"] / 1e12, 3)
        result["layer_split_tflop"] = {k: round(v / 1e12, 3)
                                       for k, v in lw.items()}
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        if layer_path:
            cb = cpu_baseline_layer(st, k_src, v_src, doc_off, x, wts, prm,
                                    args.cpu_seconds, y=step.y)
            result["parity"] = cb.pop("parity", None)
            result["cpu_baseline"] = cb
        else:
            got = None
            if score_path:
                got = {"out": step.out, "lse": step.lse, "score": step.score}
            elif not score_path:
                # one more (untimed) step that also writes the LSE; the
                # outputs are deterministic, so O and s are those timed
                step.lse = torch.empty((st.n_tokens, st.n_q_heads),
                                       dtype=torch.float32, device=dev)
                one_step()
                torch.cuda.synchronize()
                got = {"out": step.out, "lse": step.lse, "score": step.score}
            cb = cpu_baseline(st, k_src, v_src, doc_off, online, prm,
                              args.cpu_seconds, last_only=score_path,
                              family=fam, got=got)
            result["parity"] = cb.pop("parity", None)
            result["cpu_baseline"] = cb
    print(json.dumps(result), flush=True)
    par = result.get("parity")
    if par and "max_bound_ratio" in par:
        if par["max_bound_ratio"] > 1.0:
            raise SystemExit(f"layer parity beyond its bound: {par}")
    elif par and max(par["max_abs_O"], par["max_abs_s"],
                     par["max_abs_lse"] or 0.0) > PARITY_TOL:
        raise SystemExit(f"parity above {PARITY_TOL}: {par}")


if __name__ == "__main__":
    main()
