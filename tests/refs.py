"""Independent references used to pin the oracle (test helpers).

Two formulations that differ from the oracle's split prefix/own-key loops:

* ``attention_sdpa`` -- library routines only: torch ``F.rms_norm``, the
  Hugging Face Qwen3 rotary embedding (``Qwen3RotaryEmbedding`` and
  ``apply_rotary_pos_emb``, which fix the rotate-half convention and the
  theta^(-2i/D) frequencies), and ``scaled_dot_product_attention`` with
  ``enable_gqa`` (which fixes the contiguous q-head -> kv-head grouping) over
  an explicit boolean mask on the concatenated [prefix ; online] sequence.
  HF computes rotary angles from float32 inverse frequencies, so agreement is
  ~1e-5, not 1e-12.
* ``attention_concat_fp64`` -- numpy float64 brute force over the
  concatenated sequence with a plain causal mask (prefix rows precede every
  online row, so causal-over-concatenation equals "prefix fully visible +
  causal online"), RoPE as complex multiplication by exp(i * pos * freq).
"""
from __future__ import annotations

import numpy as np


def bf16_bits_to_f64(u: np.ndarray) -> np.ndarray:
    u = np.ascontiguousarray(u, dtype=np.uint16)
    return (u.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def torch_bf16_to_bits(t) -> np.ndarray:
    import torch
    return t.detach().to("cpu").contiguous().view(torch.int16).numpy().view(
        np.uint16)


def _pair_slices(prob, p):
    d = int(prob["doc_ids"][p])
    L = int(prob["doc_len"][d])
    off = int(prob["doc_off"][d])
    tok0 = int(prob["cu_seqlens"][p])
    T = int(prob["cu_seqlens"][p + 1]) - tok0
    return d, L, off, tok0, T


def attention_sdpa(prob, rms_eps=1e-6, rope_theta=1e6, scale=None):
    import torch
    import torch.nn.functional as F
    from transformers import Qwen3Config
    from transformers.models.qwen3.modeling_qwen3 import (
        Qwen3RotaryEmbedding, apply_rotary_pos_emb)

    Hq, Hkv, D = prob["n_q_heads"], prob["n_kv_heads"], prob["head_dim"]
    scale = scale if scale is not None else D ** -0.5
    cfg = Qwen3Config(head_dim=D, rope_theta=rope_theta,
                      num_attention_heads=Hq, num_key_value_heads=Hkv,
                      hidden_size=Hq * D)
    rot = Qwen3RotaryEmbedding(cfg)
    f = lambda a: torch.from_numpy(bf16_bits_to_f64(a))
    pk, pv = f(prob["prefix_k"]), f(prob["prefix_v"])
    Q, K, V = f(prob["q"]), f(prob["k"]), f(prob["v"])
    wq, wk = f(prob["q_norm_w"]), f(prob["k_norm_w"])
    out = torch.zeros(Q.shape, dtype=torch.float64)
    for p in range(len(prob["doc_ids"])):
        d, L, off, tok0, T = _pair_slices(prob, p)
        q = Q[tok0:tok0 + T].permute(1, 0, 2)[None]      # [1,Hq,T,D]
        k = K[tok0:tok0 + T].permute(1, 0, 2)[None]      # [1,Hkv,T,D]
        v = V[tok0:tok0 + T].permute(1, 0, 2)[None]
        qn = F.rms_norm(q, (D,), weight=wq, eps=rms_eps)
        kn = F.rms_norm(k, (D,), weight=wk, eps=rms_eps)
        pos = torch.arange(L, L + T)[None]
        cos, sin = rot(qn, pos)
        qr, kr = apply_rotary_pos_emb(qn, kn, cos, sin)
        kp = pk[off:off + L].permute(1, 0, 2)[None]      # [1,Hkv,L,D]
        vp = pv[off:off + L].permute(1, 0, 2)[None]
        keys = torch.cat([kp, kr], dim=2)
        vals = torch.cat([vp, v], dim=2)
        mask = torch.ones(T, L + T, dtype=torch.bool)
        mask[:, L:] = torch.tril(torch.ones(T, T, dtype=torch.bool))
        o = F.scaled_dot_product_attention(qr, keys, vals, attn_mask=mask,
                                           scale=scale, enable_gqa=True)
        out[tok0:tok0 + T] = o[0].permute(1, 0, 2)
    return out.numpy()


def attention_sdpa_llama(prob, cfg):
    """Library-routine reference for attention without QK-norm: the Hugging
    Face Llama rotary embedding (its frequencies, including the Llama-3
    rescaling of long wavelengths, come from the module's own init) and
    SDPA with GQA over the masked [prefix ; online] sequence.  Returns
    (out float64 [Ntok, Hq, D], the module's inverse frequencies float64)."""
    import torch
    import torch.nn.functional as F
    from transformers.models.llama.modeling_llama import (
        LlamaRotaryEmbedding, apply_rotary_pos_emb)

    Hq, Hkv, D = prob["n_q_heads"], prob["n_kv_heads"], prob["head_dim"]
    rot = LlamaRotaryEmbedding(cfg)
    f = lambda a: torch.from_numpy(bf16_bits_to_f64(a))
    pk, pv = f(prob["prefix_k"]), f(prob["prefix_v"])
    Q, K, V = f(prob["q"]), f(prob["k"]), f(prob["v"])
    out = torch.zeros(Q.shape, dtype=torch.float64)
    for p in range(len(prob["doc_ids"])):
        d, L, off, tok0, T = _pair_slices(prob, p)
        q = Q[tok0:tok0 + T].permute(1, 0, 2)[None]
        k = K[tok0:tok0 + T].permute(1, 0, 2)[None]
        v = V[tok0:tok0 + T].permute(1, 0, 2)[None]
        pos = torch.arange(L, L + T)[None]
        cos, sin = rot(q, pos)
        qr, kr = apply_rotary_pos_emb(q, k, cos, sin)
        kp = pk[off:off + L].permute(1, 0, 2)[None]
        vp = pv[off:off + L].permute(1, 0, 2)[None]
        keys = torch.cat([kp, kr], dim=2)
        vals = torch.cat([vp, v], dim=2)
        mask = torch.ones(T, L + T, dtype=torch.bool)
        mask[:, L:] = torch.tril(torch.ones(T, T, dtype=torch.bool))
        o = F.scaled_dot_product_attention(qr, keys, vals, attn_mask=mask,
                                           scale=D ** -0.5, enable_gqa=True)
        out[tok0:tok0 + T] = o[0].permute(1, 0, 2)
    return out.numpy(), rot.inv_freq.double().numpy()


def _rope_complex(x, pos, theta, freq=None):
    D = x.shape[-1]
    half = D // 2
    if freq is None:
        freq = theta ** (-np.arange(half, dtype=np.float64) * 2.0 / D)
    z = (x[..., :half] + 1j * x[..., half:]) * np.exp(
        1j * np.multiply.outer(pos, freq))[:, None, :]
    return np.concatenate([z.real, z.imag], axis=-1)


def _rms(x, w, eps):
    return x / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps) * w


def attention_concat_fp64(prob, rms_eps=1e-6, rope_theta=1e6, scale=None,
                          inv_freq=None):
    """Returns (out [Ntok,Hq,D], lse [Ntok,Hq]) in float64.  Without norm
    gains in prob (q_norm_w None) q and k are rotated as given; inv_freq
    overrides theta^(-2i/D)."""
    from scipy.special import logsumexp
    Hq, Hkv, D = prob["n_q_heads"], prob["n_kv_heads"], prob["head_dim"]
    rep = Hq // Hkv
    scale = scale if scale is not None else D ** -0.5
    f = bf16_bits_to_f64
    pk, pv = f(prob["prefix_k"]), f(prob["prefix_v"])
    Q, K, V = f(prob["q"]), f(prob["k"]), f(prob["v"])
    norm = prob.get("q_norm_w") is not None
    if norm:
        wq, wk = f(prob["q_norm_w"]), f(prob["k_norm_w"])
    out = np.zeros(Q.shape)
    lse = np.zeros(Q.shape[:2])
    for p in range(len(prob["doc_ids"])):
        d, L, off, tok0, T = _pair_slices(prob, p)
        pos = np.arange(L, L + T, dtype=np.float64)
        qs, ks = Q[tok0:tok0 + T], K[tok0:tok0 + T]
        if norm:
            qs, ks = _rms(qs, wq, rms_eps), _rms(ks, wk, rms_eps)
        qh = _rope_complex(qs, pos, rope_theta, inv_freq)    # [T,Hq,D]
        kh = _rope_complex(ks, pos, rope_theta, inv_freq)    # [T,Hkv,D]
        keys = np.concatenate([pk[off:off + L], kh], axis=0)  # [S,Hkv,D]
        vals = np.concatenate([pv[off:off + L], V[tok0:tok0 + T]], axis=0)
        S = L + T
        causal = np.arange(S)[None, :] <= (L + np.arange(T))[:, None]
        for h in range(Hq):
            g = h // rep
            z = scale * qh[:, h, :] @ keys[:, g, :].T         # [T,S]
            z = np.where(causal, z, -np.inf)
            m = logsumexp(z, axis=1)
            out[tok0:tok0 + T, h] = np.exp(z - m[:, None]) @ vals[:, g, :]
            lse[tok0:tok0 + T, h] = m
    return out, lse
