"""Pins of the float64 oracle against facts fixed outside it.

Each ``pin_*`` function takes an oracle library handle (the real one, or a
copy built from a deliberately broken source in the mutation test) and
raises AssertionError when the oracle disagrees with:
  * library routines (torch SDPA + F.rms_norm + Hugging Face's Qwen3 rotary
    embedding) over the concatenated [prefix ; online] sequence,
  * a float64 numpy brute force with complex-exponential RoPE,
  * closed forms (uniform logits -> mean of the visible values, lse =
    log(#keys); all-ones values -> 1; one key -> its value; RoPE's
    relative-position property),
  * invariances (pair order, duplicated documents, bad ids),
  * the paper's printed memory figures (Tables 3, 9, 13, 14),
  * Hugging Face's Llama rotary embedding + SDPA for attention without
    QK-norm and with caller-given rotary frequencies (head sizes 128, 64),
  * Python's stable sort (grouping) and torch (score head).
"""
from __future__ import annotations

import os

import numpy as np

import oracle
import refs
import workloads

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def make_problem(doc_len, doc_ids, seqlens, n_q_heads=16, n_kv_heads=8,
                 seed=0, key_scale=1.0):
    st = workloads.custom(doc_len, doc_ids, seqlens, n_q_heads, n_kv_heads)
    k_src, v_src, doc_off, _ = workloads.prefix_source(
        st, "cpu", seed * 100 + 1, key_scale)
    on = workloads.online_inputs(st, "cpu", seed * 100 + 3)
    prm = workloads.params(st, "cpu", seed * 100 + 6)
    b = refs.torch_bf16_to_bits
    return dict(
        n_q_heads=n_q_heads, n_kv_heads=n_kv_heads, head_dim=128,
        doc_len=st.doc_len, doc_ids=st.doc_ids, cu_seqlens=st.cu_seqlens,
        doc_off=doc_off, prefix_k=b(k_src), prefix_v=b(v_src),
        q=b(on["q"]), k=b(on["k"]), v=b(on["v"]),
        q_norm_w=b(prm["q_norm_w"]), k_norm_w=b(prm["k_norm_w"]),
        norm_w=b(prm["norm_w"]), w_head=b(prm["w_head"]))


def run_oracle(prob, L=None, **kw):
    return oracle.prefix_attn(
        prob["doc_ids"], prob["cu_seqlens"], prob["doc_len"], prob["doc_off"],
        prob["prefix_k"], prob["prefix_v"], prob["q"], prob["k"], prob["v"],
        prob["q_norm_w"], prob["k_norm_w"], n_q_heads=prob["n_q_heads"],
        n_kv_heads=prob["n_kv_heads"], L=L, **kw)


# Shapes small enough for the brute force, covering L = 0, 1, ragged L,
# T = 1 (score token only), repeated documents, n_rep = 1, 2, 4.
CASES = [
    dict(doc_len=[5, 0, 17, 3], doc_ids=[0, 2, 1, 3, 2],
         seqlens=[4, 1, 6, 3, 2], n_q_heads=4, n_kv_heads=2),
    dict(doc_len=[1, 9], doc_ids=[1, 0, 1], seqlens=[5, 3, 1],
         n_q_heads=2, n_kv_heads=2),
    dict(doc_len=[6, 2], doc_ids=[0, 1], seqlens=[3, 4],
         n_q_heads=8, n_kv_heads=2),
]


def pin_sdpa(L):
    for i, c in enumerate(CASES):
        prob = make_problem(**c, seed=i)
        out, _, st = run_oracle(prob, L)
        assert (st == 0).all()
        ref = refs.attention_sdpa(prob)
        err = np.abs(out - ref).max()
        assert err < 1e-5, f"case {i}: oracle vs SDPA max err {err}"


def pin_concat_fp64(L):
    for i, c in enumerate(CASES):
        prob = make_problem(**c, seed=10 + i)
        out, lse, _ = run_oracle(prob, L)
        ref, ref_lse = refs.attention_concat_fp64(prob)
        err = np.abs(out - ref).max()
        lerr = np.abs(lse - ref_lse).max()
        assert err < 1e-10 and lerr < 1e-10, (i, err, lerr)


def pin_no_prefix_is_causal_self_attention(L):
    """L_d = 0: plain causal self-attention at positions 0..T-1."""
    import torch
    import torch.nn.functional as F
    from transformers import Qwen3Config
    from transformers.models.qwen3.modeling_qwen3 import (
        Qwen3RotaryEmbedding, apply_rotary_pos_emb)
    prob = make_problem([0], [0, 0], [7, 2], 4, 2, seed=21)
    out, _, _ = run_oracle(prob, L)
    f = lambda a: torch.from_numpy(refs.bf16_bits_to_f64(a))
    rot = Qwen3RotaryEmbedding(Qwen3Config(head_dim=128, rope_theta=1e6,
                                           num_attention_heads=4,
                                           num_key_value_heads=2,
                                           hidden_size=512))
    for p in range(2):
        t0, t1 = int(prob["cu_seqlens"][p]), int(prob["cu_seqlens"][p + 1])
        q = f(prob["q"][t0:t1]).permute(1, 0, 2)[None]
        k = f(prob["k"][t0:t1]).permute(1, 0, 2)[None]
        v = f(prob["v"][t0:t1]).permute(1, 0, 2)[None]
        qn = F.rms_norm(q, (128,), f(prob["q_norm_w"]), 1e-6)
        kn = F.rms_norm(k, (128,), f(prob["k_norm_w"]), 1e-6)
        cos, sin = rot(qn, torch.arange(t1 - t0)[None])
        qr, kr = apply_rotary_pos_emb(qn, kn, cos, sin)
        ref = F.scaled_dot_product_attention(qr, kr, v, is_causal=True,
                                             enable_gqa=True)
        err = np.abs(out[t0:t1] - ref[0].permute(1, 0, 2).numpy()).max()
        assert err < 1e-5, err


def pin_uniform_logits(L):
    """q = 0 makes every logit 0: out = mean of the visible values and
    lse = log(L + j + 1), whatever the keys."""
    prob = make_problem([4, 11], [1, 0, 1], [3, 5, 2], 4, 2, seed=31)
    prob["q"] = np.zeros_like(prob["q"])
    out, lse, _ = run_oracle(prob, L)
    f = refs.bf16_bits_to_f64
    pv, v = f(prob["prefix_v"]), f(prob["v"])
    for p, d in enumerate(prob["doc_ids"]):
        Ld, off = int(prob["doc_len"][d]), int(prob["doc_off"][d])
        t0 = int(prob["cu_seqlens"][p])
        for j in range(int(prob["cu_seqlens"][p + 1]) - t0):
            vis = np.concatenate([pv[off:off + Ld], v[t0:t0 + j + 1]], 0)
            mean = vis.mean(axis=0)                     # [Hkv, D]
            exp = np.repeat(mean, 2, axis=0)            # q head h -> h // 2
            assert np.abs(out[t0 + j] - exp).max() < 1e-12
            assert np.abs(lse[t0 + j] - np.log(Ld + j + 1)).max() < 1e-12


def pin_ones_values(L):
    """Softmax weights sum to 1: all-ones values give exactly 1."""
    prob = make_problem([7, 3], [0, 1], [4, 6], 4, 2, seed=41,
                        key_scale=4.0)
    one = np.uint16(0x3F80)  # bf16 1.0
    prob["prefix_v"] = np.full_like(prob["prefix_v"], one)
    prob["v"] = np.full_like(prob["v"], one)
    out, _, _ = run_oracle(prob, L)
    assert np.abs(out - 1.0).max() < 1e-13


def pin_single_key(L):
    """L_d = 0, T = 1: the only visible key is the token's own."""
    prob = make_problem([0], [0, 0], [1, 1], 8, 2, seed=51)
    out, lse, _ = run_oracle(prob, L)
    v = refs.bf16_bits_to_f64(prob["v"])
    assert np.abs(out - np.repeat(v, 4, axis=1)).max() == 0.0
    # a single key: lse is that key's logit, finite
    assert np.isfinite(lse).all()


def pin_relative_positions(L):
    """RoPE makes own-key logits depend only on j - t, so prepending a
    prefix with zero values rescales the output by exp(lse_0 - lse_L)."""
    prob = make_problem([0, 5], [0, 1], [6, 6], 4, 2, seed=61)
    T = 6
    for name in ("q", "k", "v"):     # same online tokens in both pairs
        prob[name][T:2 * T] = prob[name][0:T]
    prob["prefix_v"] = np.zeros_like(prob["prefix_v"])
    out, lse, _ = run_oracle(prob, L)
    o0, o5 = out[:T], out[T:]
    pred = o0 * np.exp(lse[:T] - lse[T:])[..., None]
    assert np.abs(o5 - pred).max() < 1e-12


def pin_invariances(L):
    """Pairs are scored independently: permuting pairs permutes outputs,
    and a document duplicated under another id scores identically."""
    prob = make_problem([3, 9, 5], [2, 0, 1, 2, 0], [3, 1, 4, 2, 5], 4, 2,
                        seed=71)
    out, lse, _ = run_oracle(prob, L)
    cu = prob["cu_seqlens"]
    perm = [3, 0, 4, 2, 1]
    seg = lambda a, p: a[cu[p]:cu[p + 1]]
    p2 = dict(prob)
    p2["doc_ids"] = prob["doc_ids"][perm]
    lens = np.diff(cu)[perm]
    p2["cu_seqlens"] = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    for name in ("q", "k", "v"):
        p2[name] = np.concatenate([seg(prob[name], p) for p in perm])
    out2, lse2, _ = run_oracle(p2, L)
    ref = np.concatenate([seg(out, p) for p in perm])
    assert np.array_equal(out2, ref)
    assert np.array_equal(lse2, np.concatenate([seg(lse, p) for p in perm]))
    # duplicate document 2 as a new id 3 pointing at the same slots
    p3 = dict(prob)
    p3["doc_len"] = np.append(prob["doc_len"], prob["doc_len"][2])
    p3["doc_off"] = np.append(prob["doc_off"], prob["doc_off"][2])
    p3["doc_ids"] = prob["doc_ids"].copy()
    p3["doc_ids"][3] = 3
    out3, _, _ = run_oracle(p3, L)
    assert np.array_equal(out3, out)


def pin_doc_range(L):
    """Out-of-range or non-resident documents: zero outputs, lse -inf,
    status DOC_RANGE; other pairs unaffected."""
    prob = make_problem([4, -1, 6], [0, 1, 5, -2, 2], [2, 3, 1, 2, 3], 4, 2,
                        seed=81)
    out, lse, st = run_oracle(prob, L)
    assert list(st) == [0, oracle.ORACLE_DOC_RANGE, oracle.ORACLE_DOC_RANGE,
                        oracle.ORACLE_DOC_RANGE, 0]
    cu = prob["cu_seqlens"]
    for p in (1, 2, 3):
        assert (out[cu[p]:cu[p + 1]] == 0).all()
        assert np.isneginf(lse[cu[p]:cu[p + 1]]).all()
    ref, ref_lse = refs.attention_concat_fp64(
        {**prob, "doc_ids": prob["doc_ids"][[0, 4]],
         "cu_seqlens": np.array([0, 2, 5], np.int32),
         "q": np.concatenate([prob["q"][0:2], prob["q"][8:11]]),
         "k": np.concatenate([prob["k"][0:2], prob["k"][8:11]]),
         "v": np.concatenate([prob["v"][0:2], prob["v"][8:11]])})
    got = np.concatenate([out[0:2], out[8:11]])
    assert np.abs(got - ref).max() < 1e-10


def pin_score_rows(L):
    """Last-layer scoring: each pair's score-token row, against the
    brute force's last rows, then through the score head against torch;
    bad documents give zero rows and lse -inf in the pair-indexed layout."""
    import torch
    import torch.nn.functional as F
    for i, c in enumerate(CASES):
        prob = make_problem(**c, seed=30 + i)
        out, lse, st = run_oracle(prob, L, last_only=True)
        assert (st == 0).all()
        ref, ref_lse = refs.attention_concat_fp64(prob)
        last = prob["cu_seqlens"][1:] - 1
        P = len(prob["doc_ids"])
        assert out.shape == (P, prob["n_q_heads"], 128)
        assert np.abs(out - ref[last]).max() < 1e-10, i
        assert np.abs(lse - ref_lse[last]).max() < 1e-10, i
        W = prob["n_q_heads"] * 128
        prm = workloads.params(workloads.custom([1], [0], [1],
                                                prob["n_q_heads"],
                                                prob["n_kv_heads"]),
                               "cpu", 40 + i, width=W)
        nw = refs.torch_bf16_to_bits(prm["norm_w"])
        wh = refs.torch_bf16_to_bits(prm["w_head"])
        logits, s = oracle.score(out.reshape(P, W), nw, wh, 1e-6, L=L)
        hn = F.rms_norm(torch.from_numpy(ref[last].reshape(P, W)), (W,),
                        torch.from_numpy(refs.bf16_bits_to_f64(nw)), 1e-6)
        tl = F.linear(hn, torch.from_numpy(refs.bf16_bits_to_f64(wh))).numpy()
        assert np.abs(logits - tl).max() < 1e-10, i
    prob = make_problem([4, -1, 6], [0, 1, 5, -2, 2], [2, 3, 1, 2, 3], 4, 2,
                        seed=82)
    out, lse, st = run_oracle(prob, L, last_only=True)
    assert list(st) == [0, oracle.ORACLE_DOC_RANGE, oracle.ORACLE_DOC_RANGE,
                        oracle.ORACLE_DOC_RANGE, 0]
    assert (out[1:4] == 0).all() and np.isneginf(lse[1:4]).all()
    full, full_lse, _ = run_oracle(prob, L)
    last = prob["cu_seqlens"][1:] - 1
    assert np.abs(out[[0, 4]] - full[last[[0, 4]]]).max() < 1e-12


def pin_decoder_layer(L):
    """The decoder-layer oracle against Hugging Face's Qwen3DecoderLayer in
    float64 with eager attention: each pair runs alone, its document's
    prefix states injected as the layer's pre-filled cache and its online
    tokens at positions L_d + j.  HF forms rotary angles from float32
    inverse frequencies, hence the 1e-5 bound."""
    import torch
    from transformers import Qwen3Config
    from transformers.cache_utils import DynamicCache
    from transformers.models.qwen3.modeling_qwen3 import (
        Qwen3DecoderLayer, Qwen3RotaryEmbedding)
    cases = [dict(doc_len=[5, 0, 17], doc_ids=[0, 2, 1, 2], seqlens=[4, 1, 6, 3],
                  n_q_heads=4, n_kv_heads=2),
             dict(doc_len=[9, 3], doc_ids=[1, 0], seqlens=[5, 2],
                  n_q_heads=8, n_kv_heads=2)]
    W, I = 192, 320
    for ci, c in enumerate(cases):
        prob = make_problem(**c, seed=60 + ci)
        st = workloads.custom(c["doc_len"], c["doc_ids"], c["seqlens"],
                              c["n_q_heads"], c["n_kv_heads"])
        b = refs.torch_bf16_to_bits
        x = b(workloads.hidden_states(st, W, "cpu", 70 + ci))
        wts = {k: b(t) for k, t in workloads.layer_weights(
            st, W, I, "cpu", 80 + ci).items()}
        y, _, status = oracle.decoder_layer(
            x, prob["doc_ids"], prob["cu_seqlens"], prob["doc_len"],
            prob["doc_off"], prob["prefix_k"], prob["prefix_v"], wts,
            prob["q_norm_w"], prob["k_norm_w"], n_q_heads=c["n_q_heads"],
            n_kv_heads=c["n_kv_heads"], L=L)
        assert (status == 0).all()
        Hq, Hkv = c["n_q_heads"], c["n_kv_heads"]
        cfg = Qwen3Config(hidden_size=W, intermediate_size=I,
                          num_attention_heads=Hq, num_key_value_heads=Hkv,
                          head_dim=128, rope_theta=1e6, rms_norm_eps=1e-6,
                          num_hidden_layers=1)
        cfg._attn_implementation = "eager"
        layer = Qwen3DecoderLayer(cfg, layer_idx=0).double().eval()
        f = lambda a: torch.from_numpy(refs.bf16_bits_to_f64(a))
        with torch.no_grad():
            layer.input_layernorm.weight.copy_(f(wts["attn_norm"]))
            layer.self_attn.q_proj.weight.copy_(f(wts["wq"]))
            layer.self_attn.k_proj.weight.copy_(f(wts["wk"]))
            layer.self_attn.v_proj.weight.copy_(f(wts["wv"]))
            layer.self_attn.o_proj.weight.copy_(f(wts["wo"]))
            layer.self_attn.q_norm.weight.copy_(f(prob["q_norm_w"]))
            layer.self_attn.k_norm.weight.copy_(f(prob["k_norm_w"]))
            layer.post_attention_layernorm.weight.copy_(f(wts["mlp_norm"]))
            layer.mlp.gate_proj.weight.copy_(f(wts["w_gate"]))
            layer.mlp.up_proj.weight.copy_(f(wts["w_up"]))
            layer.mlp.down_proj.weight.copy_(f(wts["w_down"]))
        rot = Qwen3RotaryEmbedding(cfg)
        X = f(x)
        pk = f(prob["prefix_k"])
        pv = f(prob["prefix_v"])
        cu = prob["cu_seqlens"]
        for p in range(len(c["doc_ids"])):
            d = int(prob["doc_ids"][p])
            Ld, off = int(prob["doc_len"][d]), int(prob["doc_off"][d])
            t0, T = int(cu[p]), int(cu[p + 1] - cu[p])
            cache = DynamicCache()
            if Ld > 0:
                cache.update(pk[off:off + Ld].permute(1, 0, 2)[None].contiguous(),
                             pv[off:off + Ld].permute(1, 0, 2)[None].contiguous(),
                             0)
            hs = X[t0:t0 + T][None]
            pos = torch.arange(Ld, Ld + T)[None]
            cos, sin = rot(hs, pos)
            mask = torch.zeros(1, 1, T, Ld + T, dtype=torch.float64)
            for j in range(T):
                mask[0, 0, j, Ld + j + 1:] = -torch.inf
            with torch.no_grad():
                out = layer(hs, attention_mask=mask, position_ids=pos,
                            past_key_values=cache if Ld > 0 else None,
                            position_embeddings=(cos, sin))
            out = out[0] if isinstance(out, tuple) else out
            err = np.abs(out[0].numpy() - y[t0:t0 + T]).max()
            assert err < 1e-5, f"case {ci} pair {p}: layer vs HF {err}"


def pin_score(L):
    """Score head vs torch (F.rms_norm then a [2, W] linear map), the
    yes/no swap and the sigmoid/softmax identity."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(5)
    P, W = 9, 256
    h = rng.standard_normal((P, W)) * rng.uniform(0.1, 3.0, (P, 1))
    st = workloads.custom([1], [0], [1], 2, 2)
    prm = workloads.params(st, "cpu", 91, width=W)
    nw, wh = (refs.torch_bf16_to_bits(prm["norm_w"]),
              refs.torch_bf16_to_bits(prm["w_head"]))
    logits, s = oracle.score(h, nw, wh, 1e-6, L=L)
    th = torch.from_numpy(h)
    hn = F.rms_norm(th, (W,), torch.from_numpy(refs.bf16_bits_to_f64(nw)),
                    1e-6)
    ref = F.linear(hn, torch.from_numpy(refs.bf16_bits_to_f64(wh))).numpy()
    assert np.abs(logits - ref).max() < 1e-12
    assert np.abs(s - (ref[:, 0] - ref[:, 1])).max() < 1e-12
    _, s_sw = oracle.score(h, nw, wh[::-1], 1e-6, L=L)
    assert np.abs(s_sw + s).max() < 1e-12
    sig = 1.0 / (1.0 + np.exp(-s))
    sm = torch.softmax(torch.from_numpy(logits[:, ::-1].copy()), -1)[:, 1]
    assert np.abs(sig - sm.numpy()).max() < 1e-12


def pin_group(L):
    """Canonical grouping equals Python's stable sort on (doc id, pair)."""
    rng = np.random.default_rng(7)
    n_docs = 50
    doc_len = rng.integers(-1, 20, n_docs).astype(np.int32)
    doc_ids = rng.integers(-3, n_docs + 3, 400).astype(np.int32)
    gd, gp, po = oracle.group(doc_ids, doc_len, L=L)
    valid = [p for p in range(len(doc_ids))
             if 0 <= doc_ids[p] < n_docs and doc_len[doc_ids[p]] >= 0]
    ref = sorted(valid, key=lambda p: (doc_ids[p], p))
    assert list(po) == ref
    docs = sorted({int(doc_ids[p]) for p in valid})
    assert list(gd) == docs
    for g, d in enumerate(docs):
        members = [p for p in ref if doc_ids[p] == d]
        assert list(po[gp[g]:gp[g + 1]]) == members


def read_memory_golden():
    rows = []
    with open(os.path.join(GOLDEN, "paper_memory.txt")) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                t, model, ds, system, budget, mib = line.split()
                rows.append((t, model, ds, system, int(budget), float(mib)))
    return rows


LAYERS = {"0.6B": 28, "4B": 36, "8B": 36}


def pin_store_bytes(L):
    """Closed-form store size reproduces every printed memory figure."""
    rows = read_memory_golden()
    assert len(rows) >= 40
    for t, model, ds, system, budget, mib in rows:
        b = oracle.store_payload_bytes(LAYERS[model], 8, 128,
                                       np.array([budget], np.int32), L=L)
        assert abs(b / 2 ** 20 - mib) < 5e-3, (t, model, ds, system, b)
    # Table 13's average row: 2 subsets of 512 tokens, 10 of 1024, each
    # compressed 8x.
    full = np.array([512] * 2 + [1024] * 10, np.int32)
    tot_full = oracle.store_payload_bytes(28, 8, 128, full, L=L)
    tot_dopr = oracle.store_payload_bytes(28, 8, 128, full // 8, L=L)
    assert round(tot_full / 12 / 2 ** 20, 2) == 102.67
    assert round(tot_dopr / 12 / 2 ** 20, 2) == 12.83
    # non-resident documents hold nothing
    assert oracle.store_payload_bytes(
        1, 8, 128, np.array([-1, 0, 2], np.int32), L=L) == 2 * 4096


def _bits(x):
    """float -> bf16 bit patterns, round to nearest even (test-side)."""
    f = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return ((f + (((f >> 16) & 1) + 0x7FFF)) >> 16).astype(np.uint16)


def llama_config(n_q_heads, n_kv_heads, head_dim):
    """Llama-3-family attention settings (rope_theta 5e5 and the Llama-3
    rescaling of long rotary wavelengths, as in Llama-3.2-1B)."""
    from transformers import LlamaConfig
    return LlamaConfig(
        hidden_size=n_q_heads * head_dim, num_attention_heads=n_q_heads,
        num_key_value_heads=n_kv_heads, head_dim=head_dim,
        rope_theta=500000.0, max_position_embeddings=131072,
        rope_scaling={"rope_type": "llama3", "factor": 32.0,
                      "low_freq_factor": 1.0, "high_freq_factor": 4.0,
                      "original_max_position_embeddings": 8192})


def make_problem_nonorm(doc_len, doc_ids, seqlens, n_q_heads, n_kv_heads,
                        head_dim, seed):
    """Seeded N(0,1) bf16 inputs at any head size, with no norm gains."""
    rng = np.random.default_rng(seed)
    doc_len = np.asarray(doc_len, np.int32)
    cu = np.concatenate([[0], np.cumsum(seqlens)]).astype(np.int32)
    doc_off = np.concatenate([[0], np.cumsum(doc_len)[:-1]]).astype(np.int64)
    slots, ntok = int(doc_len.sum()), int(cu[-1])
    g = lambda *shape: _bits(rng.standard_normal(shape))
    return dict(
        n_q_heads=n_q_heads, n_kv_heads=n_kv_heads, head_dim=head_dim,
        doc_len=doc_len, doc_ids=np.asarray(doc_ids, np.int32),
        cu_seqlens=cu, doc_off=doc_off,
        prefix_k=g(max(slots, 1), n_kv_heads, head_dim)[:slots],
        prefix_v=g(max(slots, 1), n_kv_heads, head_dim)[:slots],
        q=g(ntok, n_q_heads, head_dim), k=g(ntok, n_kv_heads, head_dim),
        v=g(ntok, n_kv_heads, head_dim), q_norm_w=None, k_norm_w=None)


def pin_llama_family(L):
    """Attention without QK-norm and with the caller's rotary frequencies
    (Llama-3 family, head sizes 128 and 64): the oracle given Hugging Face's
    Llama rotary module's inverse frequencies agrees with that module plus
    SDPA (HF forms the angles in float32, hence 1e-5) and with the float64
    brute force fed the same frequencies.  The Llama-3 frequencies differ
    from theta^(-2i/D), so ignoring them cannot pass."""
    for i, (D, hq, hkv) in enumerate([(128, 8, 2), (64, 4, 1)]):
        prob = make_problem_nonorm([7, 0, 12], [2, 0, 1, 2], [5, 3, 1, 4],
                                   hq, hkv, D, seed=91 + i)
        ref, inv_freq = refs.attention_sdpa_llama(prob,
                                                  llama_config(hq, hkv, D))
        plain = 500000.0 ** (-np.arange(D // 2) * 2.0 / D)
        assert np.abs(inv_freq / plain - 1).max() > 0.5
        out, lse, st = run_oracle(prob, L, rope_theta=500000.0,
                                  rope_inv_freq=inv_freq)
        assert (st == 0).all()
        err = np.abs(out - ref).max()
        assert err < 1e-5, f"D={D}: oracle vs HF Llama rotary + SDPA {err}"
        bf, bf_lse = refs.attention_concat_fp64(prob, rope_theta=500000.0,
                                                inv_freq=inv_freq)
        assert np.abs(out - bf).max() < 1e-10
        assert np.abs(lse - bf_lse).max() < 1e-10


ALL_PINS = [pin_sdpa, pin_concat_fp64, pin_no_prefix_is_causal_self_attention,
            pin_uniform_logits, pin_ones_values, pin_single_key,
            pin_relative_positions, pin_invariances, pin_doc_range,
            pin_score_rows, pin_decoder_layer, pin_score, pin_group,
            pin_store_bytes, pin_llama_family]
