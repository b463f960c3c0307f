"""GPU-side set-up for the parity tests: seeded inputs on the device, the
HIP path through the C ABI, and the float64 oracle on the same bytes (copied
device -> host; nothing the oracle reads comes from the HIP path)."""
from __future__ import annotations

import dataclasses
import sys
import time

import numpy as np

import oracle
import refs
import workloads


def log(msg):
    print(f"[{time.strftime('%H:%M:%S')}] {msg}", flush=True)
    sys.stdout.flush()


@dataclasses.dataclass
class Case:
    st: workloads.Structure
    k_src: object
    v_src: object
    doc_off: np.ndarray      # row of each resident doc's first slot
    online: dict
    prm: dict
    store: object
    step: object
    doc_ids: object
    cu: object


def setup(st, seed=0, key_scale=1.0, kernel_variant=0, device="cuda"):
    import torch
    from paper_2609_03311_amd import pipeline
    log(f"setup {st.name}: P={st.n_pairs} Ntok={st.n_tokens} "
        f"Hq={st.n_q_heads} Hkv={st.n_kv_heads} seed={seed} "
        f"variant={kernel_variant}")
    k_src, v_src, doc_off, _ = workloads.prefix_source(
        st, device, seed * 100 + 1, key_scale)
    online = workloads.online_inputs(st, device, seed * 100 + 3)
    prm = workloads.params(st, device, seed * 100 + 6)
    store = pipeline.make_store(st.doc_len, st.n_kv_heads, k_src, v_src,
                                device=device)
    max_t = int(st.seqlens.max()) if st.n_pairs else 1
    step = pipeline.OnlineStep(store, n_pairs=st.n_pairs,
                               n_q_heads=st.n_q_heads,
                               total_tokens=st.n_tokens, max_tokens=max_t,
                               kernel_variant=kernel_variant, device=device,
                               with_lse=True)
    doc_ids = torch.from_numpy(st.doc_ids).to(device)
    cu = torch.from_numpy(st.cu_seqlens).to(device)
    torch.cuda.synchronize()
    return Case(st, k_src, v_src, doc_off, online, prm, store, step, doc_ids,
                cu)


def run(case: Case):
    import torch
    from paper_2609_03311_amd import dopr_check_status
    o = case.online
    p = case.prm
    case.step.run(0, case.doc_ids, case.cu, o["q"], o["k"], o["v"],
                  p["q_norm_w"], p["k_norm_w"], p["norm_w"], p["w_head"])
    torch.cuda.synchronize()
    return dopr_check_status(case.store)


def oracle_subset(case: Case, pairs, last_only=False):
    """Oracle outputs for a subset of pairs (in the given order); with
    last_only, only each pair's score-token row (out/lse indexed by the
    position of the pair in `pairs`)."""
    import torch
    st = case.st
    pairs = np.asarray(pairs, np.int64)
    cu = st.cu_seqlens.astype(np.int64)
    docs = np.unique(st.doc_ids[pairs])
    docs = docs[(docs >= 0) & (docs < st.n_docs)]
    docs = docs[st.doc_len[docs] >= 0]
    # prefix slots of the needed documents, copied from the generator output
    sub_off = np.full(st.n_docs, -1, np.int64)
    rows, pos = [], 0
    for d in docs:
        L = int(st.doc_len[d])
        sub_off[d] = pos
        rows.append((int(case.doc_off[d]), L))
        pos += L
    idx = np.concatenate([np.arange(o, o + L) for o, L in rows]) if rows \
        else np.zeros(0, np.int64)
    it = torch.from_numpy(idx).to(case.k_src.device)
    pk = refs.torch_bf16_to_bits(case.k_src.index_select(0, it))
    pv = refs.torch_bf16_to_bits(case.v_src.index_select(0, it))
    tok = np.concatenate([np.arange(cu[p], cu[p + 1]) for p in pairs])
    tt = torch.from_numpy(tok).to(case.k_src.device)
    q = refs.torch_bf16_to_bits(case.online["q"].index_select(0, tt))
    k = refs.torch_bf16_to_bits(case.online["k"].index_select(0, tt))
    v = refs.torch_bf16_to_bits(case.online["v"].index_select(0, tt))
    lens = (cu[pairs + 1] - cu[pairs]).astype(np.int64)
    sub_cu = np.zeros(len(pairs) + 1, np.int64)
    np.cumsum(lens, out=sub_cu[1:])
    t0 = time.time()
    out, lse, status = oracle.prefix_attn(
        st.doc_ids[pairs], sub_cu.astype(np.int32), st.doc_len, sub_off, pk,
        pv, q, k, v, refs.torch_bf16_to_bits(case.prm["q_norm_w"]),
        refs.torch_bf16_to_bits(case.prm["k_norm_w"]),
        n_q_heads=st.n_q_heads, n_kv_heads=st.n_kv_heads,
        last_only=last_only)
    h = (out if last_only else out[sub_cu[1:] - 1]).reshape(len(pairs), -1)
    logits, s = oracle.score(h, refs.torch_bf16_to_bits(case.prm["norm_w"]),
                             refs.torch_bf16_to_bits(case.prm["w_head"]))
    log(f"oracle on {len(pairs)} pairs ({len(tok)} tokens): "
        f"{time.time() - t0:.1f}s")
    return dict(tok=tok, out=out, lse=lse, status=status, logits=logits,
                score=s)


def gpu_subset(case: Case, pairs, tok):
    import torch
    dev = case.step.out.device
    tt = torch.from_numpy(np.asarray(tok, np.int64)).to(dev)
    pt = torch.from_numpy(np.asarray(pairs, np.int64)).to(dev)
    out = case.step.out.index_select(0, tt).float().cpu().numpy()
    lse = case.step.lse.index_select(0, tt).cpu().numpy()
    score = case.step.score.index_select(0, pt).cpu().numpy()
    logits = case.step.logits.index_select(0, pt).cpu().numpy()
    return dict(out=out, lse=lse, score=score, logits=logits)


TOL = 2e-2  # max-abs on O and s (bf16 inputs, fp32 accumulation)


def compare(case: Case, pairs, tol=TOL):
    ref = oracle_subset(case, pairs)
    got = gpu_subset(case, pairs, ref["tok"])
    valid = ref["status"] == 0
    e_out = float(np.abs(got["out"] - ref["out"]).max()) if got["out"].size \
        else 0.0
    fin = np.isfinite(ref["lse"])
    e_lse = float(np.abs(got["lse"][fin] - ref["lse"][fin]).max()) \
        if fin.any() else 0.0
    e_s = float(np.abs(got["score"][valid] - ref["score"][valid]).max()) \
        if valid.any() else 0.0
    e_l = float(np.abs(got["logits"][valid] - ref["logits"][valid]).max()) \
        if valid.any() else 0.0
    mean_out = float(np.abs(got["out"] - ref["out"]).mean()) \
        if got["out"].size else 0.0
    log(f"{case.st.name}: {len(pairs)} pairs max|dO|={e_out:.3e} "
        f"mean|dO|={mean_out:.3e} max|dlse|={e_lse:.3e} "
        f"max|ds|={e_s:.3e} max|dlogit|={e_l:.3e}")
    assert e_out <= tol, f"O max-abs {e_out} > {tol}"
    assert e_s <= tol, f"score max-abs {e_s} > {tol}"
    assert e_l <= tol, f"logit max-abs {e_l} > {tol}"
    assert e_lse <= tol, f"lse max-abs {e_lse} > {tol}"
    return dict(out=e_out, score=e_s, lse=e_lse)


def sample_pairs(st, n_random, seed=0, include_largest_group=True,
                 max_group=None):
    rng = np.random.default_rng(1234 + seed)
    P = st.n_pairs
    picks = set(rng.choice(P, min(n_random, P), replace=False).tolist())
    if include_largest_group and P:
        u, c = np.unique(st.doc_ids, return_counts=True)
        big = u[np.argmax(c)]
        members = np.nonzero(st.doc_ids == big)[0]
        if max_group is not None and len(members) > max_group:
            members = np.sort(rng.choice(members, max_group, replace=False))
        picks.update(members.tolist())
    picks.update([0, P - 1])
    return np.array(sorted(picks), np.int64)


def pass_strata(st, rows_per_item=2048, pass_rows=256):
    """Where each valid pair sits among the 256-row passes of its work item,
    from the canonical grouping (pairs of a document in pair order, T_p *
    n_rep stacked rows each, a group's rows cut into near-equal items on
    32-row boundaries): 0 = its first row is in the item's first pass,
    2 = its last row is in the item's last pass (and not 0), 1 = neither.
    Pairs without a valid document get -1."""
    gd, gp, order = oracle.group(st.doc_ids, st.doc_len)
    n_rep = st.n_q_heads // st.n_kv_heads
    rows = st.seqlens[order].astype(np.int64) * n_rep
    prow = np.zeros(len(order) + 1, np.int64)
    np.cumsum(rows, out=prow[1:])
    pos = np.full(st.n_pairs, -1, np.int64)
    for g in range(len(gd)):
        s0, s1 = int(gp[g]), int(gp[g + 1])
        base, R = int(prow[s0]), int(prow[s1] - prow[s0])
        n_it = -(-R // rows_per_item)
        cuts = np.array([base + ((k * R // n_it) & ~31) for k in range(n_it)]
                        + [base + R], np.int64)
        for s in range(s0, s1):
            r0, r1 = int(prow[s]), int(prow[s + 1]) - 1
            k = min(int(np.searchsorted(cuts, r0, "right")) - 1, n_it - 1)
            a, b = int(cuts[k]), int(cuts[k + 1])
            n_pass = -(-(b - a) // pass_rows)
            first = (r0 - a) // pass_rows == 0
            k1 = min(int(np.searchsorted(cuts, r1, "right")) - 1, n_it - 1)
            a1, b1 = int(cuts[k1]), int(cuts[k1 + 1])
            last = (r1 - a1) // pass_rows == -(-(b1 - a1) // pass_rows) - 1
            pos[order[s]] = 0 if first else (2 if last else 1)
    return pos


def stratified_pairs(st, per_stratum, seed=0, max_group=None):
    """per_stratum pairs (or all there are) from each pass_strata class, plus
    the most-reused document's group and the first and last pair."""
    rng = np.random.default_rng(4321 + seed)
    pos = pass_strata(st)
    picks = set()
    for c in (0, 1, 2):
        m = np.nonzero(pos == c)[0]
        if len(m):
            picks.update(rng.choice(m, min(per_stratum, len(m)),
                                    replace=False).tolist())
    picks.update(sample_pairs(st, 0, seed, max_group=max_group).tolist())
    return np.array(sorted(picks), np.int64), pos


# ---------------------------------------------------------------------------
# Last-layer scoring (score-token rows with the fused score head).

def setup_score(case: Case, kernel_variant=0, with_rows=True):
    """A ScoreStep over the same store and inputs as `case`."""
    from paper_2609_03311_amd import pipeline
    st = case.st
    max_t = int(st.seqlens.max()) if st.n_pairs else 1
    return pipeline.ScoreStep(case.store, n_pairs=st.n_pairs,
                              n_q_heads=st.n_q_heads,
                              total_tokens=st.n_tokens, max_tokens=max_t,
                              kernel_variant=kernel_variant,
                              device=case.step.out.device,
                              with_rows=with_rows)


def run_score(case: Case, sstep):
    import torch
    from paper_2609_03311_amd import dopr_check_status
    o = case.online
    p = case.prm
    sstep.run(0, case.doc_ids, case.cu, o["q"], o["k"], o["v"],
              p["q_norm_w"], p["k_norm_w"], p["norm_w"], p["w_head"])
    torch.cuda.synchronize()
    return dopr_check_status(case.store)


def compare_score(case: Case, sstep, pairs, tol=TOL):
    import torch
    ref = oracle_subset(case, pairs, last_only=True)
    pt = torch.from_numpy(np.asarray(pairs, np.int64)).to(sstep.score.device)
    got_s = sstep.score.index_select(0, pt).cpu().numpy()
    got_l = sstep.logits.index_select(0, pt).cpu().numpy()
    valid = ref["status"] == 0
    e_s = float(np.abs(got_s - ref["score"]).max()) if len(pairs) else 0.0
    e_l = float(np.abs(got_l - ref["logits"]).max()) if len(pairs) else 0.0
    e_out = e_lse = 0.0
    if sstep.out is not None:
        got_o = sstep.out.index_select(0, pt).float().cpu().numpy()
        got_lse = sstep.lse.index_select(0, pt).cpu().numpy()
        e_out = float(np.abs(got_o - ref["out"]).max()) if len(pairs) else 0.0
        fin = np.isfinite(ref["lse"])
        assert (np.isneginf(got_lse) == ~fin).all(), "lse -inf mismatch"
        e_lse = float(np.abs(got_lse[fin] - ref["lse"][fin]).max()) \
            if fin.any() else 0.0
    log(f"{case.st.name} score rows: {len(pairs)} pairs "
        f"({int(valid.sum())} valid) max|dO|={e_out:.3e} "
        f"max|dlse|={e_lse:.3e} max|ds|={e_s:.3e} max|dlogit|={e_l:.3e}")
    assert e_out <= tol, f"O max-abs {e_out} > {tol}"
    assert e_lse <= tol, f"lse max-abs {e_lse} > {tol}"
    assert e_s <= tol, f"score max-abs {e_s} > {tol}"
    assert e_l <= tol, f"logit max-abs {e_l} > {tol}"
    return dict(out=e_out, score=e_s, lse=e_lse)


# ---------------------------------------------------------------------------
# One decoder layer around the attention.

@dataclasses.dataclass
class LayerCase:
    base: Case
    x: object          # device bf16 [Ntok, W]
    weights: dict      # device bf16 tensors (generator names)
    lstep: object
    hidden: int
    inter: int


def setup_layer(case: Case, hidden=None, inter=None, seed=0,
                kernel_variant=0):
    from paper_2609_03311_amd import pipeline
    st = case.st
    W, I = workloads.layer_dims(st)
    W, I = hidden or W, inter or I
    dev = case.step.out.device
    x = workloads.hidden_states(st, W, dev, seed * 100 + 11)
    wts = workloads.layer_weights(st, W, I, dev, seed * 100 + 21)
    max_t = int(st.seqlens.max()) if st.n_pairs else 1
    lstep = pipeline.LayerStep(case.store, wts, n_pairs=st.n_pairs,
                               n_q_heads=st.n_q_heads,
                               total_tokens=st.n_tokens, max_tokens=max_t,
                               hidden=W, intermediate=I,
                               kernel_variant=kernel_variant, device=dev)
    log(f"layer {st.name}: W={W} I={I} workspace "
        f"{lstep.workspace.numel() / 2**20:.0f} MiB")
    return LayerCase(case, x, wts, lstep, W, I)


def run_layer(lc: LayerCase):
    import torch
    from paper_2609_03311_amd import dopr_check_status
    c = lc.base
    lc.lstep.run(0, c.doc_ids, c.cu, lc.x, c.prm["q_norm_w"],
                 c.prm["k_norm_w"])
    torch.cuda.synchronize()
    return dopr_check_status(c.store)


def oracle_layer_subset(lc: LayerCase, pairs):
    """The float64 layer oracle on the tokens of a subset of pairs (every
    projection is row-wise, so the subset is exact)."""
    import torch
    c = lc.base
    st = c.st
    pairs = np.asarray(pairs, np.int64)
    cu = st.cu_seqlens.astype(np.int64)
    docs = np.unique(st.doc_ids[pairs])
    docs = docs[(docs >= 0) & (docs < st.n_docs)]
    docs = docs[st.doc_len[docs] >= 0]
    sub_off = np.full(st.n_docs, -1, np.int64)
    rows, pos = [], 0
    for d in docs:
        L = int(st.doc_len[d])
        sub_off[d] = pos
        rows.append((int(c.doc_off[d]), L))
        pos += L
    idx = np.concatenate([np.arange(o, o + L) for o, L in rows]) if rows \
        else np.zeros(0, np.int64)
    dev = c.k_src.device
    it = torch.from_numpy(idx).to(dev)
    pk = refs.torch_bf16_to_bits(c.k_src.index_select(0, it))
    pv = refs.torch_bf16_to_bits(c.v_src.index_select(0, it))
    tok = np.concatenate([np.arange(cu[p], cu[p + 1]) for p in pairs])
    tt = torch.from_numpy(tok).to(dev)
    x = refs.torch_bf16_to_bits(lc.x.index_select(0, tt))
    lens = (cu[pairs + 1] - cu[pairs]).astype(np.int64)
    sub_cu = np.zeros(len(pairs) + 1, np.int64)
    np.cumsum(lens, out=sub_cu[1:])
    wts = {k: refs.torch_bf16_to_bits(v) for k, v in lc.weights.items()}
    t0 = time.time()
    y, _, status = oracle.decoder_layer(
        x, st.doc_ids[pairs], sub_cu.astype(np.int32), st.doc_len, sub_off,
        pk, pv, wts, refs.torch_bf16_to_bits(c.prm["q_norm_w"]),
        refs.torch_bf16_to_bits(c.prm["k_norm_w"]), n_q_heads=st.n_q_heads,
        n_kv_heads=st.n_kv_heads)
    log(f"layer oracle on {len(pairs)} pairs ({len(tok)} tokens): "
        f"{time.time() - t0:.1f}s")
    return dict(tok=tok, y=y, status=status)


def compare_layer(lc: LayerCase, pairs, atol, rtol):
    """|y - y_ref| <= atol + rtol |y_ref| elementwise."""
    import torch
    ref = oracle_layer_subset(lc, pairs)
    tt = torch.from_numpy(ref["tok"]).to(lc.lstep.y.device)
    got = lc.lstep.y.index_select(0, tt).float().cpu().numpy()
    err = np.abs(got - ref["y"])
    bound = atol + rtol * np.abs(ref["y"])
    worst = float((err / bound).max()) if err.size else 0.0
    rel_rms = float(np.sqrt((err ** 2).mean() / (ref["y"] ** 2).mean())) \
        if err.size else 0.0
    log(f"{lc.base.st.name} layer: {len(pairs)} pairs max|dy|="
        f"{err.max() if err.size else 0:.3e} rel-rms {rel_rms:.3e} "
        f"max|y| {np.abs(ref['y']).max() if err.size else 0:.2f} "
        f"worst err/bound {worst:.3f}")
    assert worst <= 1.0, f"layer error exceeds atol {atol} + rtol {rtol}|y|"
    return dict(max=float(err.max()) if err.size else 0.0, rel_rms=rel_rms)
