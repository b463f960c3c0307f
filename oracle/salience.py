"""Float64 oracle of offline salience selection -- TEST INFRASTRUCTURE.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this module.  It shares no code with the HIP library
and never imports it.  Plain numpy in float64; one library matrix product per
head is the only primitive.

What is computed (Sec. 3.2.1, used offline by Sec. 3.3):
  * ``mean_head_attention`` -- the document's final-layer causal
    self-attention matrix averaged over the attention (query) heads: row j
    is the attending position, column i the attended one.
  * ``salience_scores`` -- u_i, the mean of the |T_p| largest entries of
    column i, where only the causally visible entries (rows j >= i) are
    candidates, so |T_p| = min(p, n - i) with 0-based i (min(p, n - i + 1)
    in the paper's 1-based indexing).
  * ``select_top_k`` -- the K positions with the largest u.  Ties go to the
    lower position; the selected positions are returned in ascending order
    (document order), and K larger than n selects every position.
  * ``salience`` -- the three steps over a batch of documents given as the
    bf16 bit patterns of their final-layer queries and keys, exactly as they
    enter the attention product (after any norm and rotary embedding, at
    positions 0..n-1: each document is encoded on its own).
"""
from __future__ import annotations

import numpy as np


def _bf16_to_f64(u) -> np.ndarray:
    u = np.ascontiguousarray(u, dtype=np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def mean_head_attention(q, k, softmax_scale):
    """Head-averaged causal attention of one document (Sec. 3.2.1).

    q: float64 [n, Hq, D] queries, k: float64 [n, Hkv, D] keys; query head h
    reads key head h // (Hq // Hkv).  For every head the row-wise softmax of
    softmax_scale * q k^T over the visible keys i <= j; the result is the
    mean of the Hq matrices, float64 [n, n], zero above the diagonal.
    """
    n, Hq, _ = q.shape
    Hkv = k.shape[1]
    n_rep = Hq // Hkv
    visible = np.tril(np.ones((n, n), dtype=bool))
    total = np.zeros((n, n))
    for h in range(Hq):
        z = softmax_scale * (q[:, h, :] @ k[:, h // n_rep, :].T)
        z = np.where(visible, z, -np.inf)
        z = z - z.max(axis=1, keepdims=True)
        e = np.exp(z)
        total += e / e.sum(axis=1, keepdims=True)
    return total / Hq


def salience_scores(abar, p):
    """u_i = mean of the top-|T_p| values of column i among rows j >= i,
    |T_p| = min(p, n - i) (Sec. 3.2.1).  float64 [n]."""
    n = abar.shape[0]
    u = np.empty(n)
    for i in range(n):
        column = abar[i:, i]
        m = min(p, n - i)
        largest = np.sort(column)[::-1][:m]
        u[i] = largest.sum() / m
    return u


def select_top_k(u, k):
    """Positions of the k largest u (ties: lower position first), returned
    ascending; k >= len(u) selects all."""
    ranked = sorted(range(len(u)), key=lambda i: (-u[i], i))
    return np.array(sorted(ranked[:k]), dtype=np.int64)


def salience(q_bits, k_bits, cu_doclens, softmax_scale, p, n_select=None,
             docs=None, with_attention=False):
    """Salience of every token and the selected positions of every document.

    q_bits: uint16 [Ntok, Hq, D], k_bits: uint16 [Ntok, Hkv, D] (bf16 bit
    patterns); document d owns rows cu_doclens[d] .. cu_doclens[d+1]-1.
    n_select: per-document K_d (or None: no selection).  docs: subset of
    document indices to evaluate (default all).

    Returns dict(u={d: float64 [n_d]}, selected={d: int64 [K_d]},
    attention={d: float64 [n_d, n_d]} when with_attention).
    """
    cu = np.asarray(cu_doclens, dtype=np.int64)
    if docs is None:
        docs = range(len(cu) - 1)
    out = dict(u={}, selected={}, attention={})
    for d in docs:
        t0, t1 = int(cu[d]), int(cu[d + 1])
        q = _bf16_to_f64(q_bits[t0:t1])
        k = _bf16_to_f64(k_bits[t0:t1])
        abar = mean_head_attention(q, k, softmax_scale)
        u = salience_scores(abar, p)
        out["u"][d] = u
        if n_select is not None:
            out["selected"][d] = select_top_k(u, int(n_select[d]))
        if with_attention:
            out["attention"][d] = abar
    return out
