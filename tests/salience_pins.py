"""Pins of the salience oracle (Sec. 3.2.1) against facts fixed outside it.

Each ``pin_*`` raises AssertionError when the oracle module bound to the name
``salience`` disagrees with:
  * Hugging Face's Qwen3 attention (eager, float64 inputs), whose returned
    per-head attention weights, averaged over heads, are the matrix the
    paper's salience reads; the queries and keys are captured from the same
    forward, so grouping, scale and mask are HF's, not the oracle's,
  * closed forms: all-zero queries give uniform causal rows, A[j, i] =
    1/(j+1), whose column top-p means are window means of the harmonic
    sequence (exact rationals), strictly decreasing, so the top-K are the
    first K positions,
  * the special cases p = 1 (column maximum) and p >= n (column mean over
    the visible rows),
  * brute force over every subset of a tiny column,
  * numpy's stable lexsort (selection with ties),
  * the bf16 bit-pattern decoding of a few known values.
"""
from __future__ import annotations

import itertools
from fractions import Fraction

import numpy as np

from oracle import salience

D = 128


def _bits(x: np.ndarray) -> np.ndarray:
    """float -> bf16 bit patterns, round to nearest even (test-side)."""
    f = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    r = ((f >> 16) & 1) + 0x7FFF
    return ((f + r) >> 16).astype(np.uint16)


def _random_qk(n, hq, hkv, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    q = _bits(scale * rng.standard_normal((n, hq, D)))
    k = _bits(rng.standard_normal((n, hkv, D)))
    return q, k


def pin_bf16_decoding():
    v = salience._bf16_to_f64(np.array([0x3F80, 0xC000, 0x0001, 0x7F7F,
                                        0x0000, 0x8000], np.uint16))
    assert v[0] == 1.0 and v[1] == -2.0
    assert v[2] == 2.0 ** -133
    assert v[3] == (2 - 2 ** -7) * 2.0 ** 127
    assert v[4] == 0.0 and v[5] == 0.0 and np.signbit(v[5])


def pin_uniform_closed_form():
    """q = 0: every visible logit is 0, so A[j, i] = 1/(j+1) for i <= j;
    u_i = (1/m) sum_{j=i}^{i+m-1} 1/(j+1), m = min(p, n-i)."""
    for n, hq, hkv, p in [(37, 4, 2, 5), (9, 2, 2, 1), (12, 4, 1, 40),
                          (1, 2, 1, 3)]:
        _, k = _random_qk(n, hq, hkv, seed=n)
        q = np.zeros((n, hq, D), np.uint16)
        out = salience.salience(q, k, [0, n], D ** -0.5, p,
                                n_select=[min(n, 5)], with_attention=True)
        a = out["attention"][0]
        want = np.tril(np.repeat(1.0 / np.arange(1, n + 1)[:, None], n, 1))
        assert np.abs(a - want).max() < 1e-15, "uniform attention"
        for i in range(n):
            m = min(p, n - i)
            exact = sum(Fraction(1, j + 1) for j in range(i, i + m)) / m
            assert abs(out["u"][0][i] - float(exact)) < 1e-15 * n, \
                f"n={n} p={p} u[{i}]"
        assert list(out["selected"][0]) == list(range(min(n, 5)))


def pin_rows_stochastic():
    """Every row of the head-averaged causal attention sums to 1, the
    entries are non-negative and those above the diagonal are 0."""
    for n, hq, hkv, scale in [(33, 4, 2, 1.0), (20, 3, 3, 4.0),
                              (2, 8, 2, 1.0)]:
        q, k = _random_qk(n, hq, hkv, seed=100 + n, scale=scale)
        a = salience.salience(q, k, [0, n], D ** -0.5, 4,
                              with_attention=True)["attention"][0]
        assert np.abs(a.sum(axis=1) - 1.0).max() < 1e-12, "row sums"
        assert (a >= 0).all()
        assert (np.triu(a, 1) == 0).all(), "above the diagonal"


def pin_p_extremes():
    """p = 1 is the column maximum over rows j >= i; p >= n is the column
    mean over those rows."""
    n = 23
    q, k = _random_qk(n, 4, 2, seed=7, scale=2.0)
    a = salience.salience(q, k, [0, n], D ** -0.5, 1,
                          with_attention=True)["attention"][0]
    u1 = salience.salience_scores(a, 1)
    un = salience.salience_scores(a, n + 3)
    for i in range(n):
        assert u1[i] == np.max(a[i:, i])
        assert abs(un[i] - np.mean(a[i:, i])) < 1e-15


def pin_bruteforce_top_p():
    """Top-p mean equals the best mean over all m-subsets of the visible
    entries of a column (tiny lower-triangular matrices)."""
    rng = np.random.default_rng(3)
    for n in (1, 4, 7):
        a = np.tril(rng.random((n, n)))
        for p in range(1, n + 2):
            u = salience.salience_scores(a, p)
            for i in range(n):
                vis = a[i:, i]
                m = min(p, len(vis))
                best = max(sum(c) for c in itertools.combinations(vis, m))
                assert abs(u[i] - best / m) < 1e-12, f"n={n} p={p} i={i}"


def pin_select_ties():
    """Selection against numpy's stable lexsort: largest u first, ties to
    the lower position, result in ascending position order."""
    u = np.array([0.5, 0.7, 0.7, 0.1, 0.7, 0.5])
    assert list(salience.select_top_k(u, 2)) == [1, 2]
    assert list(salience.select_top_k(u, 4)) == [0, 1, 2, 4]
    assert list(salience.select_top_k(u, 0)) == []
    assert list(salience.select_top_k(u, 9)) == [0, 1, 2, 3, 4, 5]
    rng = np.random.default_rng(5)
    for n in (1, 17, 64):
        u = rng.integers(0, 4, n) / 4.0          # many ties
        for kk in (0, 1, n // 3, n):
            order = np.lexsort((np.arange(n), -u))
            want = np.sort(order[:kk])
            assert np.array_equal(salience.select_top_k(u, kk), want)


def pin_hf_attention_weights():
    """Head-averaged attention vs the per-head weights that Hugging Face's
    Qwen3 attention (eager) returns, on queries/keys captured from the same
    forward.  HF takes the softmax in float32, hence the 2e-6 bound."""
    import torch
    from transformers import Qwen3Config
    from transformers.models.qwen3 import modeling_qwen3 as m

    captured = {}
    original = m.eager_attention_forward

    def capture(module, query, key, value, attention_mask, scaling, **kw):
        captured.update(q=query, k=key, scaling=scaling)
        return original(module, query, key, value, attention_mask, scaling,
                        **kw)

    m.eager_attention_forward = capture
    try:
        for ci, (n, hq, hkv) in enumerate([(19, 8, 2), (11, 4, 4),
                                           (26, 4, 2)]):
            W = 96
            cfg = Qwen3Config(hidden_size=W, intermediate_size=64,
                              num_attention_heads=hq, num_key_value_heads=hkv,
                              head_dim=D, rope_theta=1e6, rms_norm_eps=1e-6,
                              num_hidden_layers=1)
            cfg._attn_implementation = "eager"
            torch.manual_seed(ci)
            attn = m.Qwen3Attention(cfg, layer_idx=0).double().eval()
            with torch.no_grad():
                for lin in (attn.q_proj, attn.k_proj):
                    lin.weight.normal_(0.0, 3.0 * W ** -0.5)
                attn.q_norm.weight.uniform_(0.5, 2.0)
                attn.k_norm.weight.uniform_(0.5, 2.0)
            rot = m.Qwen3RotaryEmbedding(cfg)
            x = torch.randn(1, n, W, dtype=torch.float64)
            pos = torch.arange(n)[None]
            mask = torch.triu(torch.full((n, n), -torch.inf,
                                         dtype=torch.float64), 1)[None, None]
            with torch.no_grad():
                _, w = attn(x, rot(x, pos), mask)
            q = captured["q"][0].permute(1, 0, 2).numpy()
            k = captured["k"][0].permute(1, 0, 2).numpy()
            a = salience.mean_head_attention(q, k, captured["scaling"])
            want = w[0].mean(dim=0).numpy()
            err = np.abs(a - want).max()
            assert err < 2e-6, f"case {ci}: attention vs HF {err}"
    finally:
        m.eager_attention_forward = original


def pin_batch_ragged():
    """A ragged batch gives each document what it gives alone."""
    lens = [5, 1, 12]
    cu = np.concatenate([[0], np.cumsum(lens)])
    q, k = _random_qk(int(cu[-1]), 4, 2, seed=21)
    ks = [2, 1, 12]
    batch = salience.salience(q, k, cu, D ** -0.5, 3, n_select=ks)
    for d, n in enumerate(lens):
        t0 = int(cu[d])
        alone = salience.salience(q[t0:t0 + n], k[t0:t0 + n], [0, n],
                                  D ** -0.5, 3, n_select=[ks[d]])
        assert np.array_equal(batch["u"][d], alone["u"][0])
        assert np.array_equal(batch["selected"][d], alone["selected"][0])


ALL_PINS = [pin_bf16_decoding, pin_uniform_closed_form, pin_rows_stochastic,
            pin_p_extremes, pin_bruteforce_top_p, pin_select_ties,
            pin_hf_attention_weights, pin_batch_ragged]
