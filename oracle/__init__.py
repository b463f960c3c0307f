"""Float64 CPU oracle of the DoPR online scoring step -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  It shares no code with the HIP library
(``paper_2609_03311_amd``) and never imports it.

The arithmetic lives in ``dopr_oracle.c`` (plain C, double precision, OpenMP
over pairs); this module only compiles it with gcc and marshals numpy arrays.
bf16 tensors travel as their uint16 bit patterns.

What is computed (see the C file for the step-by-step definition):
  * ``prefix_attn`` -- one layer of online attention of [q; t_score] over the
    document's injected prefix states plus causal own keys (Sec. 3.4, with the
    structured-mask semantics of Sec. 3.2.2).
  * ``score`` -- s(q,d) from the score token's state (Sec. 3.2.3).
  * ``group`` -- canonical grouping of pairs by document.
  * ``store_payload_bytes`` -- document-side prefix memory (Tables 3, 9).
  * ``decoder_layer`` -- the whole decoder layer around that attention
    (numpy, float64, in this file).
  * ``oracle.salience`` (own module, numpy float64) -- the offline salience
    selection of Sec. 3.2.1: head-averaged causal attention, column top-p
    means and the top-K positions of each document.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dopr_oracle.c")
_LIB = os.path.join(_HERE, "libdopr_oracle.so")
_lock = threading.Lock()
_lib = None

ORACLE_DOC_RANGE = -3


def build(src: str = _SRC, out: str = _LIB, extra_flags=()) -> str:
    """Compile the oracle with gcc (-O2, no fast-math) into a shared library."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared",
           "-Wall", "-Wextra", *extra_flags, "-o", out + ".tmp", src, "-lm"]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    os.replace(out + ".tmp", out)
    return out


def _bind(lib):
    P = ctypes.c_void_p
    i32, i64, f64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    lib.dopr_oracle_prefix_attn.restype = ctypes.c_int
    lib.dopr_oracle_prefix_attn.argtypes = [
        i32, i32, i32, i32, P, P, i64, P, P, P, P, P, P, P, P, P,
        f64, f64, P, f64, P, P, P, i32]
    lib.dopr_oracle_score_attn.restype = ctypes.c_int
    lib.dopr_oracle_score_attn.argtypes = lib.dopr_oracle_prefix_attn.argtypes
    lib.dopr_oracle_prefix_attn_f64.restype = ctypes.c_int
    lib.dopr_oracle_prefix_attn_f64.argtypes = \
        lib.dopr_oracle_prefix_attn.argtypes
    lib.dopr_oracle_score.restype = ctypes.c_int
    lib.dopr_oracle_score.argtypes = [i32, i32, P, P, P, f64, P, P]
    lib.dopr_oracle_group.restype = ctypes.c_int
    lib.dopr_oracle_group.argtypes = [i32, P, i64, P, P, P, P, P, P]
    lib.dopr_oracle_store_payload_bytes.restype = i64
    lib.dopr_oracle_store_payload_bytes.argtypes = [i32, i32, i32, i64, P]
    lib.dopr_oracle_max_threads.restype = ctypes.c_int
    lib.dopr_oracle_max_threads.argtypes = []
    return lib


def load_library(path: str):
    """Load (without caching) an oracle library built from some source."""
    return _bind(ctypes.CDLL(path))


def lib():
    """The oracle library, built on first use.  DOPR_ORACLE_LIB names another
    build of the same source to load instead (the sanitizer test's)."""
    global _lib
    with _lock:
        if _lib is None:
            other = os.environ.get("DOPR_ORACLE_LIB")
            if other:
                _lib = load_library(other)
                return _lib
            if not os.path.exists(_LIB) or (
                    os.path.getmtime(_LIB) < os.path.getmtime(_SRC)):
                build()
            _lib = load_library(_LIB)
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def max_threads(L=None) -> int:
    return int((L or lib()).dopr_oracle_max_threads())


def prefix_attn(doc_ids, cu_seqlens, doc_len, doc_off, prefix_k, prefix_v,
                q, k, v, q_norm_w, k_norm_w, *, n_q_heads, n_kv_heads,
                rms_eps=1e-6, rope_theta=1e6, softmax_scale=None,
                rope_inv_freq=None, threads=0, last_only=False, L=None):
    """Online prefix attention, float64.

    q_norm_w, k_norm_w: bf16 gains of the per-head RMSNorm, or both None for
    attention without QK-norm.  rope_inv_freq: float64 [D/2] rotation
    frequencies, or None for theta^(-2i/D).

    prefix_k/prefix_v: uint16 [slots, Hkv, D]; document d's slots start at
    row doc_off[d].  q: uint16 [Ntok, Hq, D]; k, v: uint16 [Ntok, Hkv, D].
    Returns (out float64 [Ntok, Hq, D], lse float64 [Ntok, Hq],
    status int32 [P]).  With last_only, only each pair's last (score) token
    is computed and out/lse are [P, Hq, D] / [P, Hq], indexed by pair.
    """
    L = L or lib()
    doc_ids = _c(doc_ids, np.int32)
    cu = _c(cu_seqlens, np.int32)
    doc_len = _c(doc_len, np.int32)
    doc_off = _c(doc_off, np.int64)
    pk = _c(prefix_k, np.uint16)
    pv = _c(prefix_v, np.uint16)
    # float64 online projections (the decoder-layer oracle) or bf16 bits
    f64 = np.asarray(q).dtype == np.float64
    qkv_t = np.float64 if f64 else np.uint16
    q = _c(q, qkv_t)
    k = _c(k, qkv_t)
    v = _c(v, qkv_t)
    assert (q_norm_w is None) == (k_norm_w is None)
    wq = None if q_norm_w is None else _c(q_norm_w, np.uint16)
    wk = None if k_norm_w is None else _c(k_norm_w, np.uint16)
    D = q.shape[-1]
    inv_freq = (None if rope_inv_freq is None
                else _c(rope_inv_freq, np.float64))
    assert inv_freq is None or inv_freq.shape == (D // 2,)
    ntok = int(cu[-1]) if cu.size else 0
    assert q.shape == (ntok, n_q_heads, D), (q.shape, ntok)
    assert k.shape == (ntok, n_kv_heads, D) and v.shape == k.shape
    if softmax_scale is None:
        softmax_scale = 1.0 / np.sqrt(D)
    P = doc_ids.shape[0]
    n_rows = P if last_only else ntok
    out = np.zeros((n_rows, n_q_heads, D), np.float64)
    lse = np.zeros((n_rows, n_q_heads), np.float64)
    status = np.zeros(P, np.int32)
    if pk.size == 0:  # keep valid pointers for documents with no slots
        pk = np.zeros((1, n_kv_heads, D), np.uint16)
        pv = np.zeros((1, n_kv_heads, D), np.uint16)
    if f64:
        assert not last_only
        fn = L.dopr_oracle_prefix_attn_f64
    else:
        fn = (L.dopr_oracle_score_attn if last_only
              else L.dopr_oracle_prefix_attn)
    rc = fn(
        P, n_q_heads, n_kv_heads, D, _p(doc_ids), _p(cu), doc_len.shape[0],
        _p(doc_len), _p(doc_off), _p(pk), _p(pv), _p(q), _p(k), _p(v),
        _p(wq) if wq is not None else None,
        _p(wk) if wk is not None else None, rms_eps, rope_theta,
        _p(inv_freq) if inv_freq is not None else None, softmax_scale,
        _p(out), _p(lse), _p(status), int(threads))
    if rc != 0:
        raise RuntimeError(f"oracle prefix_attn failed: {rc}")
    return out, lse, status


def bf16_bits_to_f64(u) -> np.ndarray:
    """Exact widening of bf16 bit patterns (the top half of an fp32)."""
    u = np.ascontiguousarray(u, dtype=np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def _rms_norm_rows(x, w, eps):
    """RMSNorm over the last axis with a gain: w * x / sqrt(mean x^2 + eps)."""
    return w * (x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps))


LAYER_WEIGHTS = ("attn_norm", "wq", "wk", "wv", "wo", "mlp_norm", "w_gate",
                 "w_up", "w_down")


def decoder_layer(x, doc_ids, cu_seqlens, doc_len, doc_off, prefix_k,
                  prefix_v, weights, q_norm_w, k_norm_w, *, n_q_heads,
                  n_kv_heads, rms_eps=1e-6, rope_theta=1e6,
                  softmax_scale=None, threads=0, L=None):
    """One decoder layer of the online pass, float64 throughout.

    Online, only the query and score tokens run through the reranker while
    every layer's attention also sees the document's stored prefix states
    (Sec. 3.4, Sec. 3.2.2); the layer is the Qwen3 decoder layer the paper
    builds on: pre-norm attention with a residual, then a pre-norm SwiGLU
    MLP with a residual.  Linear maps follow the stored-weight convention
    y = x W^T (W is [out, in]).

    x: bf16 bits [Ntok, W] entering the layer; weights: dict of bf16 bits
    attn_norm [W], wq [Hq*D, W], wk [Hkv*D, W], wv [Hkv*D, W],
    wo [W, Hq*D], mlp_norm [W], w_gate [I, W], w_up [I, W], w_down [W, I].
    Returns (y float64 [Ntok, W], attention rows float64 [Ntok, Hq, D],
    status int32 [P]).
    """
    f = bf16_bits_to_f64
    X = f(x)
    ntok, W = X.shape
    D = 128
    w = {k: f(weights[k]) for k in LAYER_WEIGHTS}
    # attention block: norm, projections, attention over [prefix ; own]
    h = _rms_norm_rows(X, w["attn_norm"], rms_eps)
    q = (h @ w["wq"].T).reshape(ntok, n_q_heads, D)
    k = (h @ w["wk"].T).reshape(ntok, n_kv_heads, D)
    v = (h @ w["wv"].T).reshape(ntok, n_kv_heads, D)
    att, _, status = prefix_attn(doc_ids, cu_seqlens, doc_len, doc_off,
                                 prefix_k, prefix_v, q, k, v, q_norm_w,
                                 k_norm_w, n_q_heads=n_q_heads,
                                 n_kv_heads=n_kv_heads, rms_eps=rms_eps,
                                 rope_theta=rope_theta,
                                 softmax_scale=softmax_scale, threads=threads,
                                 L=L)
    x2 = X + att.reshape(ntok, n_q_heads * D) @ w["wo"].T
    # MLP block: norm, gate and up projections, SiLU(gate) * up, down
    h2 = _rms_norm_rows(x2, w["mlp_norm"], rms_eps)
    g = h2 @ w["w_gate"].T
    u = h2 @ w["w_up"].T
    a = g / (1.0 + np.exp(-g)) * u
    y = x2 + a @ w["w_down"].T
    return y, att, status


def score(h, norm_w, w_head, rms_eps=1e-6, L=None):
    """Score head on float64 rows h [P, W]; returns (logits [P,2], s [P])."""
    L = L or lib()
    h = _c(h, np.float64)
    P, W = h.shape
    nw = _c(norm_w, np.uint16)
    wh = _c(w_head, np.uint16)
    assert nw.shape == (W,) and wh.shape == (2, W)
    logits = np.zeros((P, 2), np.float64)
    s = np.zeros(P, np.float64)
    rc = L.dopr_oracle_score(P, W, _p(h), _p(nw), _p(wh), rms_eps,
                             _p(logits), _p(s))
    if rc != 0:
        raise RuntimeError(f"oracle score failed: {rc}")
    return logits, s


def group(doc_ids, doc_len, L=None):
    """Canonical grouping: returns (group_doc [G], group_ptr [G+1],
    pair_order [n_valid])."""
    L = L or lib()
    doc_ids = _c(doc_ids, np.int32)
    doc_len = _c(doc_len, np.int32)
    P = doc_ids.shape[0]
    gd = np.zeros(max(P, 1), np.int32)
    gp = np.zeros(P + 1, np.int32)
    po = np.zeros(max(P, 1), np.int32)
    ng = ctypes.c_int32(0)
    nv = ctypes.c_int32(0)
    rc = L.dopr_oracle_group(P, _p(doc_ids), doc_len.shape[0], _p(doc_len),
                             ctypes.byref(ng), ctypes.byref(nv), _p(gd),
                             _p(gp), _p(po))
    if rc != 0:
        raise RuntimeError(f"oracle group failed: {rc}")
    G, V = ng.value, nv.value
    return gd[:G].copy(), gp[:G + 1].copy(), po[:V].copy()


def store_payload_bytes(n_layers, n_kv_heads, head_dim, doc_len, L=None):
    L = L or lib()
    dl = _c(doc_len, np.int32)
    return int(L.dopr_oracle_store_payload_bytes(
        n_layers, n_kv_heads, head_dim, dl.shape[0], _p(dl)))
