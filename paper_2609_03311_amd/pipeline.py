"""One decoder layer's online DoPR step on an HBM prefix store, and the
offline salience selection that decides what the store holds.

A thin convenience layer over the C ABI: it allocates device buffers with
torch and issues the library calls; all computation runs in the HIP kernels.
"""
from __future__ import annotations

import numpy as np

from . import (dopr_decoder_layer, dopr_decoder_layer_workspace,
               dopr_prefix_attn, dopr_prefix_attn_score,
               dopr_prefix_attn_score_workspace, dopr_prefix_attn_workspace,
               dopr_salience, dopr_salience_workspace, dopr_score_logits,
               dopr_store_create, dopr_store_put)

HEAD_DIM = 128


def make_store(doc_len, n_kv_heads, k_src, v_src, *, n_layers=1, layer=0,
               device="cuda", stream=None):
    """Create a store for `doc_len` and fill `layer` from canonical prefix
    states k_src/v_src [slots, Hkv, D] (bf16, device; D = 128 or 64) holding
    the resident documents' slots in ascending doc-id order."""
    import torch
    doc_len = np.ascontiguousarray(doc_len, np.int32)
    store = dopr_store_create(n_layers, n_kv_heads, int(k_src.shape[-1]),
                              doc_len, device=device, stream=stream)
    res = np.nonzero(doc_len >= 0)[0].astype(np.int32)
    if res.size:
        cu = np.zeros(res.size + 1, np.int64)
        np.cumsum(doc_len[res], out=cu[1:])
        ids = torch.from_numpy(res).to(device)
        cu_t = torch.from_numpy(cu).to(device)
        dopr_store_put(store, layer, ids, cu_t, k_src, v_src, stream=stream)
    return store


class OnlineStep:
    """Reusable buffers for the per-batch step: prefix attention over the
    store, then the score head on each pair's score-token output row."""

    def __init__(self, store, *, n_pairs, n_q_heads, total_tokens,
                 max_tokens, kernel_variant=0, device="cuda", with_lse=False,
                 rows_per_item=0, queue_order=0):
        import torch
        self.store = store
        self.n_pairs = n_pairs
        self.n_q_heads = n_q_heads
        self.total_tokens = total_tokens
        self.max_tokens = max_tokens
        self.kernel_variant = kernel_variant
        self.rows_per_item = rows_per_item
        self.queue_order = queue_order
        nbytes = dopr_prefix_attn_workspace(
            store, n_pairs=n_pairs, n_q_heads=n_q_heads,
            max_tokens=max_tokens, total_tokens=total_tokens,
            kernel_variant=kernel_variant, rows_per_item=rows_per_item)
        self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8,
                                     device=device)
        self.out = torch.empty((total_tokens, n_q_heads, store.head_dim),
                               dtype=torch.bfloat16, device=device)
        self.lse = (torch.empty((total_tokens, n_q_heads), dtype=torch.float32,
                                device=device) if with_lse else None)
        self.score = torch.empty(n_pairs, dtype=torch.float32, device=device)
        self.logits = torch.empty((n_pairs, 2), dtype=torch.float32,
                                  device=device)

    def attention(self, layer, doc_ids, cu_seqlens, q, k, v, q_norm_w,
                  k_norm_w, stream=None, **kw):
        dopr_prefix_attn(self.store, layer, doc_ids, cu_seqlens, q, k, v,
                         q_norm_w, k_norm_w, self.out, self.workspace,
                         max_tokens=self.max_tokens, lse=self.lse,
                         total_tokens=self.total_tokens,
                         kernel_variant=self.kernel_variant, stream=stream,
                         rows_per_item=self.rows_per_item,
                         **{"queue_order": self.queue_order, **kw})

    def score_head(self, cu_seqlens, norm_w, w_head, stream=None,
                   rms_eps=1e-6):
        width = self.n_q_heads * self.store.head_dim
        dopr_score_logits(self.out, norm_w, w_head, self.score, width=width,
                          h_row_stride=width, cu_seqlens=cu_seqlens,
                          logits=self.logits, rms_eps=rms_eps,
                          n_pairs=self.n_pairs, stream=stream)

    def run(self, layer, doc_ids, cu_seqlens, q, k, v, q_norm_w, k_norm_w,
            norm_w, w_head, stream=None):
        self.attention(layer, doc_ids, cu_seqlens, q, k, v, q_norm_w,
                       k_norm_w, stream=stream)
        self.score_head(cu_seqlens, norm_w, w_head, stream=stream)


class ScoreStep:
    """Reusable buffers for last-layer scoring: only each pair's score-token
    rows are attended, and the score head is fused into the attention
    epilogue.  `with_rows` keeps the rows (out [P, Hq, D], lse [P, Hq])."""

    def __init__(self, store, *, n_pairs, n_q_heads, total_tokens,
                 max_tokens, kernel_variant=0, device="cuda",
                 with_rows=True, queue_order=0):
        import torch
        self.store = store
        self.n_pairs = n_pairs
        self.n_q_heads = n_q_heads
        self.total_tokens = total_tokens
        self.max_tokens = max_tokens
        self.kernel_variant = kernel_variant
        self.queue_order = queue_order
        nbytes = dopr_prefix_attn_score_workspace(
            store, n_pairs=n_pairs, n_q_heads=n_q_heads,
            max_tokens=max_tokens, total_tokens=total_tokens,
            kernel_variant=kernel_variant)
        self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8,
                                     device=device)
        self.out = (torch.empty((n_pairs, n_q_heads, store.head_dim),
                                dtype=torch.bfloat16, device=device)
                    if with_rows else None)
        self.lse = (torch.empty((n_pairs, n_q_heads), dtype=torch.float32,
                                device=device) if with_rows else None)
        self.score = torch.empty(n_pairs, dtype=torch.float32, device=device)
        self.logits = torch.empty((n_pairs, 2), dtype=torch.float32,
                                  device=device)

    def run(self, layer, doc_ids, cu_seqlens, q, k, v, q_norm_w, k_norm_w,
            norm_w, w_head, stream=None, **kw):
        dopr_prefix_attn_score(
            self.store, layer, doc_ids, cu_seqlens, q, k, v, q_norm_w,
            k_norm_w, self.out, self.workspace, norm_w, w_head, self.score,
            max_tokens=self.max_tokens, logits=self.logits, lse=self.lse,
            total_tokens=self.total_tokens,
            kernel_variant=self.kernel_variant, stream=stream,
            **{"queue_order": self.queue_order, **kw})


# names of the layer weights in the generator's dict -> the C struct fields
LAYER_KEYS = {"attn_norm": "attn_norm_w", "wq": "w_q", "wk": "w_k",
              "wv": "w_v", "wo": "w_o", "mlp_norm": "mlp_norm_w",
              "w_gate": "w_gate", "w_up": "w_up", "w_down": "w_down"}


class LayerStep:
    """Reusable buffers for one decoder layer over the online tokens:
    x [Ntok, W] in, y [Ntok, W] out, the layer's intermediates in one
    workspace."""

    def __init__(self, store, weights, *, n_pairs, n_q_heads, total_tokens,
                 max_tokens, hidden, intermediate, kernel_variant=0,
                 device="cuda", with_lse=False):
        import torch
        self.store = store
        self.weights = {LAYER_KEYS.get(k, k): v for k, v in weights.items()}
        self.n_q_heads = n_q_heads
        self.max_tokens = max_tokens
        self.hidden = hidden
        self.intermediate = intermediate
        self.kernel_variant = kernel_variant
        nbytes = dopr_decoder_layer_workspace(
            store, self.weights, n_pairs=n_pairs, n_q_heads=n_q_heads,
            max_tokens=max_tokens, total_tokens=total_tokens, hidden=hidden,
            intermediate=intermediate, kernel_variant=kernel_variant)
        self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8,
                                     device=device)
        self.y = torch.empty((total_tokens, hidden), dtype=torch.bfloat16,
                             device=device)
        self.lse = (torch.empty((total_tokens, n_q_heads),
                                dtype=torch.float32, device=device)
                    if with_lse else None)

    def run(self, layer, doc_ids, cu_seqlens, x, q_norm_w, k_norm_w,
            stream=None, **kw):
        dopr_decoder_layer(self.store, layer, doc_ids, cu_seqlens, x, self.y,
                           self.weights, q_norm_w, k_norm_w, self.workspace,
                           n_q_heads=self.n_q_heads,
                           max_tokens=self.max_tokens, hidden=self.hidden,
                           intermediate=self.intermediate, lse=self.lse,
                           kernel_variant=self.kernel_variant, stream=stream,
                           **kw)


class SalienceStep:
    """Reusable buffers for offline salience selection of a batch of
    documents: salience u of every token and the top-K_d positions of each
    document (K_d = n_d // ratio by default).  `with_attention` keeps the
    head-averaged attention of every document ([n_docs, M, M] fp32)."""

    def __init__(self, doc_lens, *, n_q_heads, n_kv_heads, top_p,
                 n_select=None, ratio=8, max_doclen=None, device="cuda",
                 with_attention=False):
        import torch
        lens = np.asarray(doc_lens, np.int64)
        self.n_docs = int(lens.shape[0])
        self.max_doclen = int(max_doclen or max(1, int(lens.max(initial=1))))
        self.top_p = top_p
        ks = (lens // ratio if n_select is None
              else np.asarray(n_select, np.int64))
        cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
        cs = np.concatenate([[0], np.cumsum(ks)]).astype(np.int32)
        self.cu_host, self.cs_host = cu, cs
        self.cu = torch.from_numpy(cu).to(device)
        self.cs = torch.from_numpy(cs).to(device)
        ntok = int(cu[-1])
        self.u = torch.empty(ntok, dtype=torch.float32, device=device)
        self.selected = torch.empty(max(int(cs[-1]), 1), dtype=torch.int32,
                                    device=device)[:int(cs[-1])]
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        M = self.max_doclen
        self.attn_mean = (torch.empty((self.n_docs, M, M), dtype=torch.float32,
                                      device=device)
                          if with_attention else None)
        nbytes = dopr_salience_workspace(
            n_docs=self.n_docs, max_doclen=M, n_q_heads=n_q_heads,
            n_kv_heads=n_kv_heads, top_p=top_p, total_tokens=ntok,
            with_attention=with_attention)
        self.workspace = torch.empty(max(nbytes, 256), dtype=torch.uint8,
                                     device=device)

    def run(self, q, k, softmax_scale=HEAD_DIM ** -0.5, select=True,
            stream=None):
        dopr_salience(self.cu, q, k, self.u, max_doclen=self.max_doclen,
                      top_p=self.top_p, softmax_scale=softmax_scale,
                      cu_select=self.cs if select else None,
                      selected=self.selected if select else None,
                      attn_mean=self.attn_mean, status=self.status,
                      workspace=self.workspace, stream=stream)
