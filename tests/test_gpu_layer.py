"""One decoder layer of the online pass (projections, norms, SiLU gate,
residuals around the prefix attention) vs the float64 layer oracle (GPU).

Tolerance, derived from the arithmetic: every activation between steps is
stored as bf16 (relative rounding 2^-9), about six such roundings feed an
output element (h, q/k/v, the attention row, x2, h2, gate/up, SiLU*up), so
the propagated error is ~sqrt(6) * 2^-9 ~ 5e-3 of the output's scale, and
the output itself is rounded to bf16.  Elementwise:
|y - y_ref| <= 2e-2 + 2^-7 |y_ref| (four rounding units relative, an
absolute floor for small outputs), and the relative RMS error <= 1e-2.
"""
import gc

import numpy as np
import pytest

import workloads
from gpu_harness import (compare_layer, log, run_layer, sample_pairs, setup,
                         setup_layer)

pytestmark = pytest.mark.gpu

ATOL, RTOL = 2e-2, 2.0 ** -7
RMS_MAX = 1e-2


def _free():
    import torch
    gc.collect()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name,n_random", [("tiny", None),
                                           ("qwen3_0p6b", 60),
                                           ("qwen3_4b", 40),
                                           ("qwen3_8b_ragged", 12)])
def test_layer_parity(name, n_random):
    st = workloads.make(name)
    case = setup(st)
    lc = setup_layer(case)
    assert run_layer(lc) == 0
    pairs = (np.arange(st.n_pairs) if n_random is None else
             sample_pairs(st, n_random, max_group=20))
    e = compare_layer(lc, pairs, ATOL, RTOL)
    assert e["rel_rms"] <= RMS_MAX
    del case, lc
    _free()


def test_layer_shapes_and_exact_variant():
    """Ragged prefixes (L = 0, L > 256), T = 1, GQA 1 and 4, small widths,
    more tokens than one MLP chunk; the exact softmax variant agrees."""
    import torch
    rng = np.random.default_rng(5)
    P = 420
    lens = np.array([0, 7, 40, 300, 96, 97], np.int32)
    doc_ids = rng.integers(0, len(lens), P).astype(np.int32)
    seqlens = rng.choice(np.array([1, 33, 129, 200]), P).astype(np.int32)
    for hq, hkv in ((8, 8), (16, 4)):
        st = workloads.custom(lens, doc_ids, seqlens, hq, hkv,
                              name=f"layer_shapes_{hq}_{hkv}")
        case = setup(st, seed=3)
        lc = setup_layer(case, hidden=256, inter=768, seed=3)
        assert st.n_tokens > 32768        # spans two MLP chunks
        assert run_layer(lc) == 0
        e = compare_layer(lc, sample_pairs(st, 30, max_group=10), ATOL, RTOL)
        assert e["rel_rms"] <= RMS_MAX
        y0 = lc.lstep.y.clone()
        lc.lstep.kernel_variant = 4
        assert run_layer(lc) == 0
        d = (lc.lstep.y.float() - y0.float()).abs().max().item()
        log(f"{st.name}: exact vs fast softmax variant max diff {d:.3e}")
        assert d <= 0.1
        del case, lc
        _free()


def test_layer_in_place_and_bad_docs():
    """y may be x (in place) with the same bits; bad doc ids keep the layer
    running with zero attention rows (the oracle agrees) and DOC_RANGE."""
    import torch
    from paper_2609_03311_amd import DOPR_ERR_DOC_RANGE, dopr_check_status
    lens = np.array([5, -1, 9, 300], np.int32)
    st = workloads.custom(lens, [0, 1, 7, 2, -4, 3], [3, 2, 4, 1, 2, 140],
                          16, 8, name="layer_bad")
    case = setup(st, seed=11)
    lc = setup_layer(case, hidden=512, inter=1024, seed=11)
    assert run_layer(lc) == DOPR_ERR_DOC_RANGE
    compare_layer(lc, np.arange(st.n_pairs), ATOL, RTOL)
    out = lc.lstep.y.clone()
    x_keep = lc.x.clone()
    lc.lstep.y = lc.x                     # in place: y aliases x
    assert run_layer(lc) == DOPR_ERR_DOC_RANGE
    assert torch.equal(lc.x, out)
    lc.x = x_keep
    assert dopr_check_status(case.store) == 0
    _free()
