"""Python binding of libdopr (the DoPR online scoring hot path on MI355X).

Argument marshalling only: every step runs in the HIP kernels behind the C
ABI of ``include/dopr.h``; torch provides device memory and streams.  The
function names are the C names.  A non-OK status raises ``DoprError``.  If
the shared library has not been built, every call raises (there is no
fallback path).
"""
from __future__ import annotations

import ctypes
import os
from typing import Optional

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdopr.so")

DOPR_OK = 0
DOPR_ERR_INVALID_ARG = -1
DOPR_ERR_UNSUPPORTED = -2
DOPR_ERR_DOC_RANGE = -3
DOPR_ERR_WORKSPACE = -4
DOPR_ERR_HIP = -5
DOPR_ERR_SEQLEN = -6


class DoprError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class _StoreDesc(ctypes.Structure):
    _fields_ = [("n_layers", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("n_docs", ctypes.c_int64),
                ("doc_len", ctypes.c_void_p)]


class _AttnArgs(ctypes.Structure):
    _fields_ = [("n_pairs", ctypes.c_int32), ("n_q_heads", ctypes.c_int32),
                ("max_tokens", ctypes.c_int32),
                ("kernel_variant", ctypes.c_int32),
                ("total_tokens", ctypes.c_int64),
                ("doc_ids", ctypes.c_void_p), ("cu_seqlens", ctypes.c_void_p),
                ("q", ctypes.c_void_p), ("k", ctypes.c_void_p),
                ("v", ctypes.c_void_p), ("q_norm_w", ctypes.c_void_p),
                ("k_norm_w", ctypes.c_void_p), ("rms_eps", ctypes.c_float),
                ("rope_theta", ctypes.c_float),
                ("softmax_scale", ctypes.c_float), ("out", ctypes.c_void_p),
                ("lse", ctypes.c_void_p), ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t),
                ("timing_begin", ctypes.c_void_p),
                ("timing_end", ctypes.c_void_p),
                ("rope_inv_freq", ctypes.c_void_p),
                ("rows_per_item", ctypes.c_int32),
                ("queue_order", ctypes.c_int32)]


class _ScoreArgs(ctypes.Structure):
    _fields_ = [("n_pairs", ctypes.c_int32), ("width", ctypes.c_int32),
                ("h", ctypes.c_void_p), ("h_row_stride", ctypes.c_int64),
                ("row_index", ctypes.c_void_p),
                ("cu_seqlens", ctypes.c_void_p), ("norm_w", ctypes.c_void_p),
                ("w_head", ctypes.c_void_p), ("rms_eps", ctypes.c_float),
                ("logits", ctypes.c_void_p), ("score", ctypes.c_void_p)]


class _LayerArgs(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("intermediate", ctypes.c_int32),
                ("attn_norm_w", ctypes.c_void_p), ("w_q", ctypes.c_void_p),
                ("w_k", ctypes.c_void_p), ("w_v", ctypes.c_void_p),
                ("w_o", ctypes.c_void_p), ("mlp_norm_w", ctypes.c_void_p),
                ("w_gate", ctypes.c_void_p), ("w_up", ctypes.c_void_p),
                ("w_down", ctypes.c_void_p), ("x", ctypes.c_void_p),
                ("y", ctypes.c_void_p)]


class _ScoreHead(ctypes.Structure):
    _fields_ = [("norm_w", ctypes.c_void_p), ("w_head", ctypes.c_void_p),
                ("rms_eps", ctypes.c_float), ("logits", ctypes.c_void_p),
                ("score", ctypes.c_void_p)]


class _SalienceArgs(ctypes.Structure):
    _fields_ = [("n_docs", ctypes.c_int32), ("max_doclen", ctypes.c_int32),
                ("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("top_p", ctypes.c_int32), ("softmax_scale", ctypes.c_float),
                ("total_tokens", ctypes.c_int64),
                ("total_select", ctypes.c_int64),
                ("cu_doclens", ctypes.c_void_p), ("cu_select", ctypes.c_void_p),
                ("q", ctypes.c_void_p), ("k", ctypes.c_void_p),
                ("u", ctypes.c_void_p), ("selected", ctypes.c_void_p),
                ("attn_mean", ctypes.c_void_p), ("status", ctypes.c_void_p),
                ("workspace", ctypes.c_void_p),
                ("workspace_bytes", ctypes.c_size_t)]


EXPORTS = {
    "dopr_store_bytes": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p],
                         ctypes.c_int),
    "dopr_store_create": ([ctypes.c_void_p, ctypes.c_void_p, ctypes.c_size_t,
                           ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dopr_store_put": ([ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                        ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                        ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dopr_store_destroy": ([ctypes.c_void_p], ctypes.c_int),
    "dopr_store_copy_docs": ([ctypes.c_void_p, ctypes.c_void_p,
                              ctypes.c_void_p], ctypes.c_int),
    "dopr_prefix_attn_workspace": ([ctypes.c_void_p, ctypes.c_void_p,
                                    ctypes.c_void_p], ctypes.c_int),
    "dopr_prefix_attn": ([ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                          ctypes.c_void_p], ctypes.c_int),
    "dopr_prefix_attn_noalloc": ([ctypes.c_void_p, ctypes.c_int32,
                                  ctypes.c_void_p, ctypes.c_void_p],
                                 ctypes.c_int),
    "dopr_score_logits": ([ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dopr_prefix_attn_score_workspace": ([ctypes.c_void_p, ctypes.c_void_p,
                                          ctypes.c_void_p], ctypes.c_int),
    "dopr_prefix_attn_score": ([ctypes.c_void_p, ctypes.c_int32,
                                ctypes.c_void_p, ctypes.c_void_p,
                                ctypes.c_void_p], ctypes.c_int),
    "dopr_decoder_layer_workspace": ([ctypes.c_void_p, ctypes.c_void_p,
                                      ctypes.c_void_p, ctypes.c_void_p],
                                     ctypes.c_int),
    "dopr_decoder_layer": ([ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                            ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dopr_group_pairs": ([ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                          ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
                          ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                          ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dopr_gather_prefix": ([ctypes.c_void_p, ctypes.c_int32, ctypes.c_int32,
                            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                            ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dopr_salience_workspace": ([ctypes.c_void_p, ctypes.c_void_p],
                                ctypes.c_int),
    "dopr_salience": ([ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dopr_select_top_k": ([ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dopr_check_status": ([ctypes.c_void_p, ctypes.c_void_p], ctypes.c_int),
    "dopr_status_str": ([ctypes.c_int], ctypes.c_char_p),
    "dopr_last_error": ([], ctypes.c_char_p),
}

_lib = None


def lib():
    """Load libdopr.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                f"{LIB_PATH} is missing: build it with "
                "`python -m paper_2609_03311_amd._build` (no fallback exists)")
        L = ctypes.CDLL(LIB_PATH)
        for name, (argtypes, restype) in EXPORTS.items():
            fn = getattr(L, name)
            fn.argtypes = argtypes
            fn.restype = restype
        _lib = L
    return _lib


def _check(status: int):
    if status != DOPR_OK:
        L = lib()
        msg = L.dopr_last_error().decode() or L.dopr_status_str(status).decode()
        raise DoprError(status, msg)


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _desc(n_layers, n_kv_heads, head_dim, doc_len):
    import numpy as np
    dl = np.ascontiguousarray(doc_len, dtype=np.int32)
    d = _StoreDesc(n_layers, n_kv_heads, head_dim, dl.shape[0],
                   dl.ctypes.data_as(ctypes.c_void_p))
    return d, dl


def dopr_store_bytes(n_layers: int, n_kv_heads: int, head_dim: int,
                     doc_len):
    """Returns (pool_bytes, payload_bytes) for a store (host arithmetic)."""
    d, keep = _desc(n_layers, n_kv_heads, head_dim, doc_len)
    pool = ctypes.c_size_t(0)
    payload = ctypes.c_size_t(0)
    _check(lib().dopr_store_bytes(ctypes.byref(d), ctypes.byref(pool),
                                  ctypes.byref(payload)))
    return pool.value, payload.value


class Store:
    """Handle of a prefix store laid out in a caller-owned device pool."""

    def __init__(self, handle, pool, n_layers, n_kv_heads, doc_len,
                 head_dim=128):
        self.handle = handle
        self.pool = pool  # keeps the device memory alive
        self.n_layers = n_layers
        self.n_kv_heads = n_kv_heads
        self.head_dim = head_dim
        self.doc_len = doc_len

    def close(self):
        if self.handle:
            _check(lib().dopr_store_destroy(self.handle))
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def dopr_store_create(n_layers: int, n_kv_heads: int, head_dim: int,
                      doc_len, pool=None, stream=None, device=None) -> Store:
    """Create a store.  `pool` is a uint8 CUDA tensor of at least
    dopr_store_bytes(...)[0] bytes; allocated with torch if omitted."""
    import torch
    pool_bytes, _ = dopr_store_bytes(n_layers, n_kv_heads, head_dim, doc_len)
    if pool is None:
        pool = torch.empty(max(pool_bytes, 256), dtype=torch.uint8,
                           device=device or "cuda")
    d, keep = _desc(n_layers, n_kv_heads, head_dim, doc_len)
    h = ctypes.c_void_p(0)
    _check(lib().dopr_store_create(ctypes.byref(d), pool.data_ptr(),
                                   pool.numel() * pool.element_size(),
                                   _stream(stream), ctypes.byref(h)))
    return Store(h.value, pool, n_layers, n_kv_heads, keep.copy(),
                 head_dim=head_dim)


def dopr_store_put(store: Store, layer: int, doc_ids, src_cu_slots, k_src,
                   v_src, stream=None):
    _check(lib().dopr_store_put(store.handle, layer, doc_ids.numel(),
                                _ptr(doc_ids), _ptr(src_cu_slots),
                                _ptr(k_src), _ptr(v_src), _stream(stream)))


def dopr_store_destroy(store: Store):
    store.close()


def dopr_store_copy_docs(dst: Store, src: Store, stream=None):
    """Copy the documents resident in both stores (same slot counts) from
    src to dst: all layers, heads and key-norm bounds."""
    _check(lib().dopr_store_copy_docs(dst.handle, src.handle,
                                      _stream(stream)))


def _attn_args(store, doc_ids, cu_seqlens, q, k, v, q_norm_w, k_norm_w, out,
               lse, workspace, *, max_tokens, total_tokens=None,
               rms_eps=1e-6, rope_theta=1e6, softmax_scale=None,
               kernel_variant=0, timing=None, rope_inv_freq=None,
               rows_per_item=0, queue_order=0):
    n_q_heads = q.shape[1] if q is not None else store.n_kv_heads
    if total_tokens is None:
        total_tokens = q.shape[0]
    if softmax_scale is None:
        softmax_scale = store.head_dim ** -0.5
    ws_bytes = 0 if workspace is None else (
        workspace.numel() * workspace.element_size())
    return _AttnArgs(doc_ids.numel(), n_q_heads, int(max_tokens),
                     int(kernel_variant), int(total_tokens), _ptr(doc_ids),
                     _ptr(cu_seqlens), _ptr(q), _ptr(k), _ptr(v),
                     _ptr(q_norm_w), _ptr(k_norm_w), float(rms_eps),
                     float(rope_theta), float(softmax_scale), _ptr(out),
                     _ptr(lse), _ptr(workspace), ws_bytes,
                     *(timing if timing is not None else (None, None)),
                     _ptr(rope_inv_freq), int(rows_per_item),
                     int(queue_order))


def _shape_args(n_pairs, n_q_heads, max_tokens, total_tokens,
                kernel_variant, rows_per_item=0):
    a = _AttnArgs()
    a.rows_per_item = rows_per_item
    a.n_pairs = n_pairs
    a.n_q_heads = n_q_heads
    a.max_tokens = max_tokens
    a.total_tokens = total_tokens
    a.kernel_variant = kernel_variant
    a.rms_eps, a.rope_theta, a.softmax_scale = 1e-6, 1e6, 128 ** -0.5
    return a


def dopr_prefix_attn_workspace(store: Store, *, n_pairs, n_q_heads,
                               max_tokens, total_tokens,
                               kernel_variant=0, rows_per_item=0) -> int:
    a = _shape_args(n_pairs, n_q_heads, max_tokens, total_tokens,
                    kernel_variant, rows_per_item)
    n = ctypes.c_size_t(0)
    _check(lib().dopr_prefix_attn_workspace(store.handle, ctypes.byref(a),
                                            ctypes.byref(n)))
    return n.value


def dopr_prefix_attn_score_workspace(store: Store, *, n_pairs, n_q_heads,
                                     max_tokens, total_tokens,
                                     kernel_variant=0) -> int:
    a = _shape_args(n_pairs, n_q_heads, max_tokens, total_tokens,
                    kernel_variant)
    n = ctypes.c_size_t(0)
    _check(lib().dopr_prefix_attn_score_workspace(
        store.handle, ctypes.byref(a), ctypes.byref(n)))
    return n.value


def dopr_prefix_attn(store: Store, layer: int, doc_ids, cu_seqlens, q, k, v,
                     q_norm_w, k_norm_w, out, workspace, *, max_tokens,
                     lse=None, total_tokens=None, rms_eps=1e-6,
                     rope_theta=1e6, softmax_scale=None, kernel_variant=0,
                     timing=None, rope_inv_freq=None, stream=None,
                     rows_per_item=0, queue_order=0):
    """`timing` is an optional (begin, end) pair of raw hipEvent_t handles
    recorded around the attention kernel.  q_norm_w and k_norm_w may both
    be None (no QK-norm); rope_inv_freq is an optional fp32 [D/2] device
    tensor of rotation frequencies; rows_per_item 0 is the automatic work
    item size; queue_order 0/1/2 is the automatic, natural or
    longest-first order of the work queues."""
    a = _attn_args(store, doc_ids, cu_seqlens, q, k, v, q_norm_w, k_norm_w,
                   out, lse, workspace, max_tokens=max_tokens,
                   total_tokens=total_tokens, rms_eps=rms_eps,
                   rope_theta=rope_theta, softmax_scale=softmax_scale,
                   kernel_variant=kernel_variant, timing=timing,
                   rope_inv_freq=rope_inv_freq, rows_per_item=rows_per_item,
                   queue_order=queue_order)
    _check(lib().dopr_prefix_attn(store.handle, layer, ctypes.byref(a),
                                  _stream(stream)))


def dopr_prefix_attn_noalloc(store: Store, layer: int, doc_ids, cu_seqlens,
                             q, k, v, q_norm_w, k_norm_w, out, *, max_tokens,
                             lse=None, total_tokens=None, rms_eps=1e-6,
                             rope_theta=1e6, softmax_scale=None,
                             kernel_variant=0, timing=None,
                             rope_inv_freq=None, stream=None, queue_order=0):
    """dopr_prefix_attn without a workspace: the plan goes to the library's
    own per-device scratch (at most DOPR_NOALLOC_SCRATCH_BYTES)."""
    a = _attn_args(store, doc_ids, cu_seqlens, q, k, v, q_norm_w, k_norm_w,
                   out, lse, None, max_tokens=max_tokens,
                   total_tokens=total_tokens, rms_eps=rms_eps,
                   rope_theta=rope_theta, softmax_scale=softmax_scale,
                   kernel_variant=kernel_variant, timing=timing,
                   rope_inv_freq=rope_inv_freq, queue_order=queue_order)
    _check(lib().dopr_prefix_attn_noalloc(store.handle, layer,
                                          ctypes.byref(a), _stream(stream)))


DOPR_NOALLOC_SCRATCH_BYTES = 64 << 20


def dopr_prefix_attn_score(store: Store, layer: int, doc_ids, cu_seqlens, q,
                           k, v, q_norm_w, k_norm_w, out, workspace, norm_w,
                           w_head, score, *, max_tokens, logits=None,
                           lse=None, total_tokens=None, rms_eps=1e-6,
                           head_rms_eps=1e-6, rope_theta=1e6,
                           softmax_scale=None, kernel_variant=0, timing=None,
                           rope_inv_freq=None, stream=None, queue_order=0):
    """Last-layer scoring: the score token's attention rows (out [P, Hq, D]
    or None, lse [P, Hq] or None) with the score head fused (score [P],
    logits [P, 2] or None)."""
    a = _attn_args(store, doc_ids, cu_seqlens, q, k, v, q_norm_w, k_norm_w,
                   out, lse, workspace, max_tokens=max_tokens,
                   total_tokens=total_tokens, rms_eps=rms_eps,
                   rope_theta=rope_theta, softmax_scale=softmax_scale,
                   kernel_variant=kernel_variant, timing=timing,
                   rope_inv_freq=rope_inv_freq, queue_order=queue_order)
    h = _ScoreHead(_ptr(norm_w), _ptr(w_head), float(head_rms_eps),
                   _ptr(logits), _ptr(score))
    _check(lib().dopr_prefix_attn_score(store.handle, layer, ctypes.byref(a),
                                        ctypes.byref(h), _stream(stream)))


_LAYER_FIELDS = ("attn_norm_w", "w_q", "w_k", "w_v", "w_o", "mlp_norm_w",
                 "w_gate", "w_up", "w_down")


def _layer_args(weights, x, y, hidden, intermediate):
    """weights: dict with the _LAYER_FIELDS keys (device bf16 tensors)."""
    return _LayerArgs(int(hidden), int(intermediate),
                      *[_ptr(weights[k]) for k in _LAYER_FIELDS],
                      _ptr(x), _ptr(y))


def dopr_decoder_layer_workspace(store: Store, weights, *, n_pairs,
                                 n_q_heads, max_tokens, total_tokens,
                                 hidden, intermediate,
                                 kernel_variant=0) -> int:
    a = _shape_args(n_pairs, n_q_heads, max_tokens, total_tokens,
                    kernel_variant)
    la = _layer_args(weights, None, None, hidden, intermediate)
    n = ctypes.c_size_t(0)
    _check(lib().dopr_decoder_layer_workspace(
        store.handle, ctypes.byref(a), ctypes.byref(la), ctypes.byref(n)))
    return n.value


def dopr_decoder_layer(store: Store, layer: int, doc_ids, cu_seqlens, x, y,
                       weights, q_norm_w, k_norm_w, workspace, *, n_q_heads,
                       max_tokens, hidden, intermediate, lse=None,
                       rms_eps=1e-6, rope_theta=1e6, softmax_scale=None,
                       kernel_variant=0, timing=None, stream=None):
    """One decoder layer over the online tokens: x -> y ([Ntok, W] bf16)."""
    if softmax_scale is None:
        softmax_scale = 128 ** -0.5
    ws_bytes = workspace.numel() * workspace.element_size()
    a = _AttnArgs(doc_ids.numel(), int(n_q_heads), int(max_tokens),
                  int(kernel_variant), int(x.shape[0]), _ptr(doc_ids),
                  _ptr(cu_seqlens), None, None, None, _ptr(q_norm_w),
                  _ptr(k_norm_w), float(rms_eps), float(rope_theta),
                  float(softmax_scale), None, _ptr(lse), _ptr(workspace),
                  ws_bytes, *(timing if timing is not None else (None, None)))
    la = _layer_args(weights, x, y, hidden, intermediate)
    _check(lib().dopr_decoder_layer(store.handle, layer, ctypes.byref(a),
                                    ctypes.byref(la), _stream(stream)))


def dopr_score_logits(h, norm_w, w_head, score, *, width=None,
                      h_row_stride=None, row_index=None, cu_seqlens=None,
                      logits=None, rms_eps=1e-6, n_pairs=None, stream=None):
    if width is None:
        width = norm_w.numel()
    if h_row_stride is None:
        h_row_stride = width
    if n_pairs is None:
        n_pairs = score.numel()
    a = _ScoreArgs(int(n_pairs), int(width), _ptr(h), int(h_row_stride),
                   _ptr(row_index), _ptr(cu_seqlens), _ptr(norm_w),
                   _ptr(w_head), float(rms_eps), _ptr(logits), _ptr(score))
    _check(lib().dopr_score_logits(ctypes.byref(a), _stream(stream)))


def dopr_group_pairs(store: Store, doc_ids, workspace, stream=None):
    """Canonical grouping (synchronises): returns (group_doc, group_ptr,
    pair_order) as CUDA int32 tensors of their exact lengths."""
    import torch
    P = doc_ids.numel()
    dev = doc_ids.device
    gd = torch.empty(max(P, 1), dtype=torch.int32, device=dev)
    gp = torch.empty(P + 1, dtype=torch.int32, device=dev)
    po = torch.empty(max(P, 1), dtype=torch.int32, device=dev)
    ng, nv = ctypes.c_int32(0), ctypes.c_int32(0)
    _check(lib().dopr_group_pairs(
        store.handle, P, _ptr(doc_ids), _ptr(workspace),
        workspace.numel() * workspace.element_size(), ctypes.byref(ng),
        ctypes.byref(nv), _ptr(gd), _ptr(gp), _ptr(po), _stream(stream)))
    return gd[:ng.value], gp[:ng.value + 1], po[:nv.value]


def dopr_gather_prefix(store: Store, layer: int, doc_ids, out_cu_slots,
                       k_out, v_out, stream=None):
    _check(lib().dopr_gather_prefix(store.handle, layer, doc_ids.numel(),
                                    _ptr(doc_ids), _ptr(out_cu_slots),
                                    _ptr(k_out), _ptr(v_out),
                                    _stream(stream)))


def _salience_args(n_docs, max_doclen, n_q_heads, n_kv_heads, top_p,
                   softmax_scale, total_tokens, total_select, cu_doclens,
                   cu_select, q, k, u, selected, attn_mean, status, workspace):
    return _SalienceArgs(
        n_docs, max_doclen, n_q_heads, n_kv_heads, top_p, softmax_scale,
        total_tokens, total_select, _ptr(cu_doclens), _ptr(cu_select),
        _ptr(q), _ptr(k), _ptr(u), _ptr(selected), _ptr(attn_mean),
        _ptr(status), _ptr(workspace),
        0 if workspace is None else workspace.numel() * workspace.element_size())


def dopr_salience_workspace(*, n_docs, max_doclen, n_q_heads, n_kv_heads,
                            top_p, total_tokens, with_attention=False) -> int:
    """Workspace bytes of dopr_salience (shape arguments only)."""
    a = _salience_args(n_docs, max_doclen, n_q_heads, n_kv_heads, top_p,
                       1.0, total_tokens, 0, None, None, None, None, None,
                       None, None, None, None)
    if with_attention:
        a.attn_mean = 16  # any aligned non-NULL value: only its presence counts
    n = ctypes.c_size_t(0)
    _check(lib().dopr_salience_workspace(ctypes.byref(a), ctypes.byref(n)))
    return n.value


def dopr_salience(cu_doclens, q, k, u, *, max_doclen, top_p, softmax_scale,
                  cu_select=None, selected=None, attn_mean=None, status=None,
                  workspace=None, stream=None):
    """Salience of every token (and the top-K positions of each document when
    `selected` is given).  cu_doclens/cu_select: int32 device tensors;
    q [Ntok, Hq, 128], k [Ntok, Hkv, 128] bf16; u fp32 [Ntok]."""
    n_docs = cu_doclens.numel() - 1
    total_select = 0 if selected is None else selected.numel()
    a = _salience_args(n_docs, max_doclen, q.shape[1], k.shape[1], top_p,
                       softmax_scale, q.shape[0], total_select, cu_doclens,
                       cu_select, q, k, u, selected, attn_mean, status,
                       workspace)
    _check(lib().dopr_salience(ctypes.byref(a), _stream(stream)))


def dopr_select_top_k(cu_doclens, cu_select, u, selected, *, max_doclen,
                      status=None, stream=None):
    """Top-K_d positions of each document on caller-given u."""
    a = _salience_args(cu_doclens.numel() - 1, max_doclen, 1, 1, 1, 1.0,
                       u.numel(), selected.numel(), cu_doclens, cu_select,
                       None, None, u, selected, None, status, None)
    _check(lib().dopr_select_top_k(ctypes.byref(a), _stream(stream)))


def dopr_check_status(store: Store, stream=None) -> int:
    """Synchronise and return the deferred device status (0 = OK); does not
    raise so tests can inspect the code."""
    return int(lib().dopr_check_status(store.handle, _stream(stream)))


def dopr_status_str(status: int) -> str:
    return lib().dopr_status_str(status).decode()


def dopr_last_error() -> str:
    return lib().dopr_last_error().decode()
