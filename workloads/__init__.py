"""Seeded synthetic workloads for the DoPR online scoring step.

Input generators only: this module holds none of the method's arithmetic and
imports neither the oracle nor the HIP library; both are fed from here.

The shapes follow the paper's evaluation settings: Qwen3 backbones with bf16
inference (Table 7), prefix budgets of K_infer = doc_len / 8 slots (Table 8:
256/512/2048-token documents -> 32/64/256 slots) and ~100 first-stage
candidates per query.  The paper's datasets (TREC DL, BEIR, BRIGHT) and
weights are not used: seeded random states of the same shapes stand in for
them, since to the attention step the stored prefix states are opaque
already-final keys and values.

Integer structure (doc ids, prefix lengths, token counts) uses one fresh
``numpy.random.default_rng(seed)`` per workload, drawn in a fixed order.
Values are standard normal (gains 1 + 0.1 N(0,1), head weights N(0, 1/W)),
rounded to bf16, drawn with ``torch.Generator`` on the requested device in
fixed-size chunks so a given seed always yields the same bytes on a device.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, Optional

import numpy as np

HEAD_DIM = 128


@dataclasses.dataclass
class Structure:
    """Integer structure of one batch of (query, document) pairs."""
    name: str
    n_q_heads: int
    n_kv_heads: int
    hidden: int
    doc_len: np.ndarray          # int32 [n_docs]; -1 = not resident
    doc_ids: np.ndarray          # int32 [P]
    seqlens: np.ndarray          # int32 [P]: T_p = query tokens + 1 score token
    head_dim: int = HEAD_DIM
    n_layers: int = 1
    seed: int = 0

    @property
    def n_pairs(self) -> int:
        return int(self.doc_ids.shape[0])

    @property
    def n_docs(self) -> int:
        return int(self.doc_len.shape[0])

    @property
    def cu_seqlens(self) -> np.ndarray:
        cu = np.zeros(self.n_pairs + 1, np.int64)
        np.cumsum(self.seqlens, out=cu[1:])
        return cu.astype(np.int32)

    @property
    def n_tokens(self) -> int:
        return int(self.seqlens.astype(np.int64).sum())

    @property
    def n_rep(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    def resident_docs(self) -> np.ndarray:
        """Resident doc ids in ascending order (the prefix source order)."""
        return np.nonzero(self.doc_len >= 0)[0].astype(np.int32)

    def unique_docs(self) -> np.ndarray:
        return np.unique(self.doc_ids)


def _zipf_draws(rng, n_ids: int, n_draws: int, s: float) -> np.ndarray:
    """Finite Zipf: P(rank k) ~ k^-s over k = 1..n_ids by inverse CDF; the
    rank -> id map is a permutation drawn first so hot ids are scattered."""
    perm = rng.permutation(n_ids)
    w = np.arange(1, n_ids + 1, dtype=np.float64) ** (-s)
    cdf = np.cumsum(w)
    cdf /= cdf[-1]
    ranks = np.searchsorted(cdf, rng.random(n_draws), side="right")
    ranks = np.minimum(ranks, n_ids - 1)
    return perm[ranks].astype(np.int32)


def _per_query_candidates(rng, n_queries, n_docs, per_query):
    ids = [rng.choice(n_docs, per_query, replace=False)
           for _ in range(n_queries)]
    return np.concatenate(ids).astype(np.int32)


def tiny(seed: int = 0) -> Structure:
    """1 layer, 16q/8kv heads; 8 docs x 16 slots; 4 queries x (15+1)
    tokens, each paired with all 8 docs (32 pairs, query-major)."""
    n_docs, n_q = 8, 4
    doc_ids = np.array([j for _ in range(n_q) for j in range(n_docs)],
                       np.int32)
    return Structure("tiny", 16, 8, 16 * HEAD_DIM,
                     np.full(n_docs, 16, np.int32), doc_ids,
                     np.full(doc_ids.shape[0], 16, np.int32), seed=seed)


def qwen3_0p6b(seed: int = 0) -> Structure:
    """Qwen3-0.6B-shaped layer (hidden 1024, 16q/8kv): 10k docs x 32 slots
    (256-token passages at 8x); 64 queries x 100 distinct uniform docs;
    31 query tokens + score token."""
    rng = np.random.default_rng(seed)
    doc_ids = _per_query_candidates(rng, 64, 10_000, 100)
    return Structure("qwen3_0p6b", 16, 8, 1024,
                     np.full(10_000, 32, np.int32), doc_ids,
                     np.full(doc_ids.shape[0], 32, np.int32), seed=seed)


def qwen3_4b(seed: int = 0) -> Structure:
    """Qwen3-4B-shaped layer (hidden 2560, 32q/8kv): 100k docs x 64 slots;
    4096 pairs with Zipf(1.1) doc reuse; query 8-64 tokens + score token."""
    rng = np.random.default_rng(seed)
    n_docs, P = 100_000, 4096
    doc_ids = _zipf_draws(rng, n_docs, P, 1.1)
    seqlens = (rng.integers(8, 65, P) + 1).astype(np.int32)
    return Structure("qwen3_4b", 32, 8, 2560, np.full(n_docs, 64, np.int32),
                     doc_ids, seqlens, seed=seed)


def qwen3_8b(seed: int = 0) -> Structure:
    """Qwen3-8B-shaped layer (hidden 4096, 32q/8kv): 20k long docs x 256
    slots (2048-token docs at 8x); 256 queries x 100 distinct uniform docs;
    128 query tokens + score token."""
    rng = np.random.default_rng(seed)
    doc_ids = _per_query_candidates(rng, 256, 20_000, 100)
    return Structure("qwen3_8b", 32, 8, 4096, np.full(20_000, 256, np.int32),
                     doc_ids, np.full(doc_ids.shape[0], 129, np.int32),
                     seed=seed)


def llama3_8b(seed: int = 0) -> Structure:
    """Llama-3-8B-shaped attention (hidden 4096, 32q/8kv, head size 128, no
    QK-norm): the pair structure of qwen3_8b (the cross-family check runs
    the same batch through the other family's attention)."""
    st = qwen3_8b(seed)
    st.name = "llama3_8b"
    return st


def llama3_2_1b(seed: int = 0) -> Structure:
    """Llama-3.2-1B-shaped attention (hidden 2048, 32q/8kv, head size 64,
    no QK-norm; the model of the paper's cross-family check): the pair
    structure of qwen3_8b."""
    st = qwen3_8b(seed)
    st.name = "llama3_2_1b"
    st.hidden = 2048
    st.head_dim = 64
    return st


def qwen3_8b_ragged(seed: int = 0, prefix_scale: int = 1) -> Structure:
    """Qwen3-8B-shaped layer, ragged: prefix lengths uniform 8..256 slots
    over a 1M-id space; 16384 pairs, half Zipf(1.1) reuse and half distinct
    ids not in the Zipf half, shuffled; query 16..128 tokens + score token.
    Only referenced docs are resident (the full id space would exceed one
    GPU's HBM).  prefix_scale=8 gives the uncompressed comparison (each
    prefix 8x longer, same pairs)."""
    rng = np.random.default_rng(seed)
    n_ids, P = 1_000_000, 16_384
    lens = rng.integers(8, 257, n_ids).astype(np.int64)
    zipf_half = _zipf_draws(rng, n_ids, P // 2, 1.1)
    rest = np.setdiff1d(np.arange(n_ids), zipf_half, assume_unique=False)
    uniq_half = rng.choice(rest, P // 2, replace=False).astype(np.int32)
    doc_ids = np.concatenate([zipf_half, uniq_half])
    doc_ids = doc_ids[rng.permutation(P)].astype(np.int32)
    seqlens = (rng.integers(16, 129, P) + 1).astype(np.int32)
    doc_len = np.full(n_ids, -1, np.int32)
    used = np.unique(doc_ids)
    doc_len[used] = (lens[used] * prefix_scale).astype(np.int32)
    name = "qwen3_8b_ragged" + ("" if prefix_scale == 1 else
                                f"_x{prefix_scale}")
    return Structure(name, 32, 8, 4096, doc_len, doc_ids, seqlens, seed=seed)


def with_prefix_budget(st: Structure, k_infer: int) -> Structure:
    """The same pairs with every resident document's prefix set to k_infer
    slots: one inference prefix budget of a K_infer sweep (Sec. 4.5: the
    budget is chosen at deployment without retraining)."""
    doc_len = np.where(st.doc_len >= 0, k_infer, -1).astype(np.int32)
    return Structure(f"{st.name}_k{k_infer}", st.n_q_heads, st.n_kv_heads,
                     st.hidden, doc_len, st.doc_ids.copy(),
                     st.seqlens.copy(), seed=st.seed)


CONFIGS = {
    "tiny": tiny,
    "qwen3_0p6b": qwen3_0p6b,
    "qwen3_4b": qwen3_4b,
    "qwen3_8b": qwen3_8b,
    "qwen3_8b_ragged": qwen3_8b_ragged,
    "qwen3_8b_ragged_x8": lambda seed=0: qwen3_8b_ragged(seed, 8),
    "llama3_8b": llama3_8b,
    "llama3_2_1b": llama3_2_1b,
}


def make(name: str, seed: int = 0) -> Structure:
    return CONFIGS[name](seed)


def custom(doc_len, doc_ids, seqlens, n_q_heads=16, n_kv_heads=8,
           name="custom", head_dim=HEAD_DIM) -> Structure:
    """A hand-shaped structure (edge cases, sweeps)."""
    return Structure(name, int(n_q_heads), int(n_kv_heads),
                     int(n_q_heads) * int(head_dim),
                     np.asarray(doc_len, np.int32),
                     np.asarray(doc_ids, np.int32),
                     np.asarray(seqlens, np.int32), head_dim=int(head_dim))


# ---------------------------------------------------------------------------
# Values (torch; imported lazily so the integer part needs only numpy)

_CHUNK_ELEMS = 1 << 28  # values are drawn in chunks of this many elements


def _randn_bf16(shape, seed: int, device, scale: float = 1.0,
                offset: float = 0.0):
    import torch
    n = int(np.prod(shape)) if len(shape) else 1
    out = torch.empty(n, dtype=torch.bfloat16, device=device)
    gen = torch.Generator(device=device)
    for c, start in enumerate(range(0, n, _CHUNK_ELEMS)):
        stop = min(n, start + _CHUNK_ELEMS)
        gen.manual_seed(seed * 1_000_003 + c)
        x = torch.randn(stop - start, generator=gen, device=device,
                        dtype=torch.float32)
        if scale != 1.0:
            x.mul_(scale)
        if offset != 0.0:
            x.add_(offset)
        out[start:stop] = x.to(torch.bfloat16)
    return out.view(*shape)


def prefix_source(st: Structure, device="cpu", seed: int = 1,
                  key_scale: float = 1.0):
    """Canonical prefix states of every resident doc, in ascending doc-id
    order: returns (k_src, v_src) bf16 [slots, Hkv, D] and slot offsets
    doc_off int64 [n_docs] (row of each doc's first slot; -1 if not
    resident) and cu_slots int64 [n_resident+1]."""
    res = st.resident_docs()
    lens = st.doc_len[res].astype(np.int64)
    cu = np.zeros(res.shape[0] + 1, np.int64)
    np.cumsum(lens, out=cu[1:])
    doc_off = np.full(st.n_docs, -1, np.int64)
    doc_off[res] = cu[:-1]
    slots = int(cu[-1])
    shape = (slots, st.n_kv_heads, st.head_dim)
    k_src = _randn_bf16(shape, seed, device, scale=key_scale)
    v_src = _randn_bf16(shape, seed + 1, device)
    return k_src, v_src, doc_off, cu


def online_inputs(st: Structure, device="cpu", seed: int = 3) -> Dict:
    """Raw (pre-norm, pre-RoPE) online q/k/v of every pair's tokens."""
    n = st.n_tokens
    return {
        "q": _randn_bf16((n, st.n_q_heads, st.head_dim), seed, device),
        "k": _randn_bf16((n, st.n_kv_heads, st.head_dim), seed + 1, device),
        "v": _randn_bf16((n, st.n_kv_heads, st.head_dim), seed + 2, device),
    }


def params(st: Structure, device="cpu", seed: int = 6,
           width: Optional[int] = None) -> Dict:
    """Per-layer weights: QK-norm gains, score-head norm gain and yes/no
    rows.  width defaults to Hq * D (the score token's attention output row
    stands in for its hidden state in a one-layer benchmark)."""
    W = width or st.n_q_heads * st.head_dim
    D = st.head_dim
    return {
        "q_norm_w": _randn_bf16((D,), seed, device, 0.1, 1.0),
        "k_norm_w": _randn_bf16((D,), seed + 1, device, 0.1, 1.0),
        "norm_w": _randn_bf16((W,), seed + 2, device, 0.1, 1.0),
        "w_head": _randn_bf16((2, W), seed + 3, device, 1.0 / np.sqrt(W)),
    }


# Hidden and MLP widths of the Qwen3 decoder layers the workloads are shaped
# after (a small pair for the tiny case).
LAYER_DIMS = {
    "tiny": (512, 1024),
    "qwen3_0p6b": (1024, 3072),
    "qwen3_4b": (2560, 9728),
    "qwen3_8b": (4096, 12288),
    "qwen3_8b_ragged": (4096, 12288),
    "qwen3_8b_ragged_x8": (4096, 12288),
}


def layer_dims(st: Structure):
    """(hidden, intermediate) of the decoder layer for a workload."""
    base = st.name.split("_x")[0] if st.name.startswith("qwen3_8b") else \
        st.name
    return LAYER_DIMS.get(base, LAYER_DIMS["tiny"])


def hidden_states(st: Structure, hidden: int, device="cpu",
                  seed: int = 11):
    """Hidden states of the online tokens entering a layer, N(0, 1)."""
    return _randn_bf16((st.n_tokens, hidden), seed, device)


def layer_weights(st: Structure, hidden: int, intermediate: int,
                  device="cpu", seed: int = 21) -> Dict:
    """One decoder layer's weights in the [out, in] convention: the two
    norm gains 1 + 0.1 N(0,1); every projection N(0, 1/in), so activations
    stay of order one through the layer."""
    hq = st.n_q_heads * st.head_dim
    hk = st.n_kv_heads * st.head_dim
    W, I = hidden, intermediate
    return {
        "attn_norm": _randn_bf16((W,), seed, device, 0.1, 1.0),
        "wq": _randn_bf16((hq, W), seed + 1, device, W ** -0.5),
        "wk": _randn_bf16((hk, W), seed + 2, device, W ** -0.5),
        "wv": _randn_bf16((hk, W), seed + 3, device, W ** -0.5),
        "wo": _randn_bf16((W, hq), seed + 4, device, hq ** -0.5),
        "mlp_norm": _randn_bf16((W,), seed + 5, device, 0.1, 1.0),
        "w_gate": _randn_bf16((I, W), seed + 6, device, W ** -0.5),
        "w_up": _randn_bf16((I, W), seed + 7, device, W ** -0.5),
        "w_down": _randn_bf16((W, I), seed + 8, device, I ** -0.5),
    }


# ---------------------------------------------------------------------------
# Offline salience selection: batches of documents encoded on their own.
# Document lengths follow the paper's corpora at the three backbone sizes
# (256-, 512- and 2048-token documents, K_infer = n / 8 slots kept, Table 8);
# the final-layer queries and keys as they enter attention are standard
# normal bf16 (an RMS-normed, rotated head vector has entries of order one),
# so the scaled logits are N(0, q_scale^2).
SALIENCE_BATCHES = {
    # name: (document length, documents per batch, Hq, Hkv)
    "qwen3_0p6b_docs": (256, 512, 16, 8),
    "qwen3_4b_docs": (512, 256, 32, 8),
    "qwen3_8b_docs": (2048, 64, 32, 8),
}
SALIENCE_TOP_P = 8          # the paper gives no value for p
SALIENCE_RATIO = 8          # K_d = n_d / 8 (Table 8)


def salience_batch(name: str):
    """(doc_lens int32 [n_docs], Hq, Hkv) of a named salience batch."""
    n, docs, hq, hkv = SALIENCE_BATCHES[name]
    return np.full(docs, n, np.int32), hq, hkv


def salience_inputs(doc_lens, n_q_heads, n_kv_heads, device="cpu",
                    seed: int = 31, q_scale: float = 1.0):
    """Final-layer queries [Ntok, Hq, D] and keys [Ntok, Hkv, D], bf16."""
    ntok = int(np.asarray(doc_lens, np.int64).sum())
    q = _randn_bf16((ntok, n_q_heads, HEAD_DIM), seed, device, q_scale)
    k = _randn_bf16((ntok, n_kv_heads, HEAD_DIM), seed + 1, device)
    return q, k
