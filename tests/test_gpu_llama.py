"""Attention without QK-norm and with caller-given rotary frequencies (the
Llama family used for the paper's cross-family check; Appendix,
"Generalization Across Model Families"), GPU vs the float64 oracle.

Shapes are Llama-3-8B-like (32 q / 8 kv heads, head size 128) and
Llama-3.2-1B-like (the same heads at head size 64, the model the paper
checks), rope_theta 5e5 with the Llama-3 rescaling of long wavelengths; the
frequencies come from Hugging Face's Llama rotary module and reach both
sides as inputs.
Without QK-norm no logit bound is known in advance, so every work unit runs
the reference-free softmax and rows it cannot serve are recomputed by the
exact pass: the large-query case checks that hand-off against exact mode.
Tolerance: the same max-abs 2e-2 as the Qwen3 path (bf16 operands, fp32
accumulation).
"""
import numpy as np
import pytest

import oracle
import refs
import workloads
from gpu_harness import log
from oracle_pins import llama_config

pytestmark = pytest.mark.gpu

TOL = 2e-2
HEAD_SIZES = [128, 64]


def _inv_freq(hq, hkv, d):
    from transformers.models.llama.modeling_llama import LlamaRotaryEmbedding
    return LlamaRotaryEmbedding(llama_config(hq, hkv, d)).inv_freq.float()


def _case(name, doc_len, doc_ids, seqlens, hq=32, hkv=8, q_scale=1.0,
          seed=0, d=128):
    import torch
    from paper_2609_03311_amd import pipeline
    st = workloads.custom(doc_len, doc_ids, seqlens, hq, hkv, name=name,
                          head_dim=d)
    log(f"setup {name}: D={d} P={st.n_pairs} Ntok={st.n_tokens} "
        f"q_scale={q_scale}")
    k_src, v_src, doc_off, _ = workloads.prefix_source(st, "cuda",
                                                       seed * 100 + 1)
    on = workloads.online_inputs(st, "cuda", seed * 100 + 3)
    if q_scale != 1.0:
        on["q"] = (on["q"].float() * q_scale).to(torch.bfloat16)
    store = pipeline.make_store(st.doc_len, hkv, k_src, v_src)
    inv = _inv_freq(hq, hkv, d)
    return dict(st=st, k_src=k_src, v_src=v_src, doc_off=doc_off, on=on,
                store=store, inv=inv, inv_dev=inv.cuda(),
                doc_ids=torch.from_numpy(st.doc_ids).cuda(),
                cu=torch.from_numpy(st.cu_seqlens).cuda())


def _gpu(c, variant=0):
    import torch
    from paper_2609_03311_amd import dopr_check_status, pipeline
    st = c["st"]
    step = pipeline.OnlineStep(c["store"], n_pairs=st.n_pairs,
                               n_q_heads=st.n_q_heads,
                               total_tokens=st.n_tokens,
                               max_tokens=int(st.seqlens.max()),
                               kernel_variant=variant, with_lse=True)
    step.attention(0, c["doc_ids"], c["cu"], c["on"]["q"], c["on"]["k"],
                   c["on"]["v"], None, None, rope_theta=5e5,
                   rope_inv_freq=c["inv_dev"])
    torch.cuda.synchronize()
    assert dopr_check_status(c["store"]) == 0
    return step.out.float().cpu().numpy(), step.lse.cpu().numpy()


def _oracle(c, last_only=False):
    st = c["st"]
    b = refs.torch_bf16_to_bits
    return oracle.prefix_attn(
        st.doc_ids, st.cu_seqlens, st.doc_len, c["doc_off"], b(c["k_src"]),
        b(c["v_src"]), b(c["on"]["q"]), b(c["on"]["k"]), b(c["on"]["v"]),
        None, None, n_q_heads=st.n_q_heads, n_kv_heads=st.n_kv_heads,
        rope_theta=5e5, rope_inv_freq=c["inv"].double().numpy(),
        last_only=last_only)


CASES = [
    # ragged prefixes incl. L = 0 and 256, T = 1 (score token only), reuse
    ("llama_ragged", [256, 0, 33, 100, 7], [0, 2, 1, 3, 0, 4, 2],
     [129, 40, 1, 17, 64, 33, 5]),
    # one document shared by many pairs (stacked rows over several items)
    ("llama_shared", [64], [0] * 20, [65] * 20),
]


@pytest.mark.parametrize("d", HEAD_SIZES)
@pytest.mark.parametrize("name,doc_len,doc_ids,seqlens", CASES,
                         ids=[c[0] for c in CASES])
def test_no_qk_norm_parity(name, doc_len, doc_ids, seqlens, d):
    c = _case(name, doc_len, doc_ids, seqlens, d=d)
    out, lse = _gpu(c)
    ref, ref_lse, status = _oracle(c)
    assert (status == 0).all()
    e = float(np.abs(out - ref).max())
    el = float(np.abs(lse - ref_lse).max())
    log(f"{name} D={d}: max|dO|={e:.3e} max|dlse|={el:.3e}")
    assert e <= TOL and el <= TOL
    # the frequencies matter: with theta^(-2i/D) the outputs move by more
    # than the tolerance (the Llama-3 rescaling only touches the long
    # wavelengths, which turn little at these positions, so not by much)
    plain, _, _ = oracle.prefix_attn(
        c["st"].doc_ids, c["st"].cu_seqlens, c["st"].doc_len, c["doc_off"],
        refs.torch_bf16_to_bits(c["k_src"]),
        refs.torch_bf16_to_bits(c["v_src"]),
        refs.torch_bf16_to_bits(c["on"]["q"]),
        refs.torch_bf16_to_bits(c["on"]["k"]),
        refs.torch_bf16_to_bits(c["on"]["v"]), None, None,
        n_q_heads=32, n_kv_heads=8, rope_theta=5e5)
    assert float(np.abs(plain - ref).max()) > 2 * TOL


@pytest.mark.parametrize("d", HEAD_SIZES)
def test_no_qk_norm_score_rows(d):
    """Last-layer scoring without QK-norm: the score-token rows."""
    import torch
    from paper_2609_03311_amd import dopr_check_status, pipeline
    c = _case("llama_score", *CASES[0][1:], d=d)
    st = c["st"]
    prm = workloads.params(st, "cuda", 6)
    ss = pipeline.ScoreStep(c["store"], n_pairs=st.n_pairs,
                            n_q_heads=st.n_q_heads,
                            total_tokens=st.n_tokens,
                            max_tokens=int(st.seqlens.max()), with_rows=True)
    ss.run(0, c["doc_ids"], c["cu"], c["on"]["q"], c["on"]["k"],
           c["on"]["v"], None, None, prm["norm_w"], prm["w_head"],
           rope_theta=5e5, rope_inv_freq=c["inv_dev"])
    torch.cuda.synchronize()
    assert dopr_check_status(c["store"]) == 0
    ref, _, status = _oracle(c, last_only=True)
    got = ss.out.float().cpu().numpy()
    e = float(np.abs(got - ref).max())
    _, s = oracle.score(ref.reshape(st.n_pairs, -1),
                        refs.torch_bf16_to_bits(prm["norm_w"]),
                        refs.torch_bf16_to_bits(prm["w_head"]))
    es = float(np.abs(ss.score.cpu().numpy() - s).max())
    log(f"llama score rows D={d}: max|dO|={e:.3e} max|ds|={es:.3e}")
    assert (status == 0).all() and e <= TOL and es <= TOL


@pytest.mark.parametrize("d", HEAD_SIZES)
def test_no_qk_norm_large_queries_take_exact_pass(d):
    """Queries scaled x40 push the largest logits of many rows past what the
    reference-free mode represents (2^|logit| overflows): those units must be
    recomputed by the exact pass.  With |q| ~ 450 the bf16 rounding of q^
    alone moves logits by ~1, so the result is checked against exact mode
    (same operands) and for finiteness rather than against float64."""
    import torch
    c = _case("llama_large_q", [96, 200], [0, 1, 0], [20, 9, 33],
              q_scale=40.0, seed=5, d=d)
    fast, fast_lse = _gpu(c, variant=0)
    exact, exact_lse = _gpu(c, variant=4)
    assert np.isfinite(fast).all() and np.isfinite(fast_lse).all()
    d = float(np.abs(fast - exact).max())
    dl = float(np.abs(fast_lse - exact_lse).max())
    log(f"large q: fast vs exact-mode max diff O {d:.3e} lse {dl:.3e}; "
        f"max lse {float(np.abs(exact_lse).max()):.1f}")
    assert d <= TOL and dl <= 1e-3 * float(np.abs(exact_lse).max()) + TOL


def test_one_norm_gain_is_rejected():
    """Both gains or neither: a lone gain is an argument error, reported
    before anything is launched."""
    import torch
    from paper_2609_03311_amd import DOPR_ERR_INVALID_ARG, DoprError
    c = _case("llama_args", [8], [0], [4])
    st = c["st"]
    from paper_2609_03311_amd import pipeline
    step = pipeline.OnlineStep(c["store"], n_pairs=1, n_q_heads=32,
                               total_tokens=st.n_tokens, max_tokens=4)
    w = torch.ones(128, dtype=torch.bfloat16, device="cuda")
    with pytest.raises(DoprError) as e:
        step.attention(0, c["doc_ids"], c["cu"], c["on"]["q"], c["on"]["k"],
                       c["on"]["v"], w, None)
    assert e.value.status == DOPR_ERR_INVALID_ARG
