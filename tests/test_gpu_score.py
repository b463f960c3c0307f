"""Last-layer scoring (score-token rows, fused score head) vs the float64
oracle (GPU).

The oracle computes each pair's score-token row with the plain attention
loops restricted to j = T_p - 1, then the plain score head on that row.
Tolerance as for the full path: max-abs 2e-2 on O (bf16), the LSE, the
yes/no logits and s.  The kernel must also reproduce, bit for bit, the rows
the full path computes for the same tokens (same operands, same chunk
order); its fused head sums the same bf16 row in a different order than
the separate score kernel, so the two scores agree to fp32 rounding.
"""
import gc

import numpy as np
import pytest

import workloads
from gpu_harness import (compare_score, log, run, run_score, sample_pairs,
                         setup, setup_score)

pytestmark = pytest.mark.gpu


def _free():
    import torch
    gc.collect()
    torch.cuda.empty_cache()


CONFIG_CASES = [
    ("tiny", None, None),
    ("qwen3_0p6b", None, None),
    ("qwen3_4b", 300, None),           # + all 579 pairs of the hottest doc
    ("qwen3_8b", 400, None),
    ("qwen3_8b_ragged", 300, 200),
    ("qwen3_8b_ragged_x8", 100, 60),
]


@pytest.mark.parametrize("name,n_random,max_group", CONFIG_CASES,
                         ids=[c[0] for c in CONFIG_CASES])
def test_score_config_parity(name, n_random, max_group):
    st = workloads.make(name)
    case = setup(st)
    ss = setup_score(case)
    assert run_score(case, ss) == 0
    pairs = (np.arange(st.n_pairs) if n_random is None else
             sample_pairs(st, n_random, max_group=max_group))
    compare_score(case, ss, pairs)
    del case, ss
    _free()


@pytest.mark.parametrize("name", ["tiny", "qwen3_0p6b", "qwen3_4b"])
def test_score_rows_equal_full_path_rows(name):
    import torch
    st = workloads.make(name)
    case = setup(st)
    assert run(case) == 0
    ss = setup_score(case)
    assert run_score(case, ss) == 0
    last = torch.from_numpy(st.cu_seqlens[1:].astype(np.int64) - 1).cuda()
    full_o = case.step.out.index_select(0, last)
    full_lse = case.step.lse.index_select(0, last)
    diff = (full_o.float() - ss.out.float()).abs().max().item()
    assert torch.equal(full_o, ss.out), f"rows differ by {diff}"
    assert torch.equal(full_lse, ss.lse)
    ds = (case.step.score - ss.score).abs().max().item()
    dl = (case.step.logits - ss.logits).abs().max().item()
    log(f"{name}: fused vs separate score head max diff {ds:.3e} "
        f"(logits {dl:.3e})")
    assert ds < 1e-4 and dl < 1e-4
    del case, ss
    _free()


EDGE = [
    # (Hq, Hkv, prefix lengths, pairs, token counts)
    (16, 8, [0, 1, 31, 32, 33, 255, 256, 257], 30, [1, 2, 33, 129]),
    (8, 8, [0, 5, 130], 10, [1, 50, 129]),
    (8, 2, [3, 70, 600], 9, [2, 31, 65]),
    (32, 8, [2048, 300, 0], 6, [129, 7, 1]),
]


@pytest.mark.parametrize("variant", [0, 2, 4, 5])
@pytest.mark.parametrize("i", range(len(EDGE)))
def test_score_edge_shapes(i, variant):
    """Empty prefixes and prefixes longer than the resident segment (L = 0,
    L > 96, L > 256), T = 1, GQA ratios 1, 4 and 16 q heads per kv head, in
    the automatic shape (two blocks per CU), the 8-wave shape, and the exact
    and self-check variants."""
    Hq, Hkv, lens, P, Ts = EDGE[i]
    rng = np.random.default_rng(300 + i)
    doc_ids = rng.integers(0, len(lens), P).astype(np.int32)
    seqlens = rng.choice(np.asarray(Ts), P).astype(np.int32)
    st = workloads.custom(np.asarray(lens, np.int32), doc_ids, seqlens, Hq,
                          Hkv, name=f"score_edge{i}")
    case = setup(st, seed=40 + i)
    ss = setup_score(case, kernel_variant=variant)
    assert run_score(case, ss) == 0
    compare_score(case, ss, np.arange(st.n_pairs))
    del case, ss
    _free()


def test_score_bad_doc_ids():
    import torch
    from paper_2609_03311_amd import DOPR_ERR_DOC_RANGE, dopr_check_status
    lens = np.array([5, -1, 9], np.int32)       # doc 1 not resident
    st = workloads.custom(lens, [0, 1, 7, 2, -4], [3, 2, 4, 1, 2], 16, 8,
                          name="score_bad")
    case = setup(st, seed=11)
    ss = setup_score(case)
    ss.out.fill_(7.0)
    ss.lse.fill_(7.0)
    ss.score.fill_(7.0)
    ss.logits.fill_(7.0)
    assert run_score(case, ss) == DOPR_ERR_DOC_RANGE
    for p in (1, 2, 4):
        assert (ss.out[p] == 0).all()
        assert torch.isneginf(ss.lse[p]).all()
        assert ss.score[p].item() == 0 and (ss.logits[p] == 0).all()
    compare_score(case, ss, np.arange(st.n_pairs))
    assert dopr_check_status(case.store) == 0
    _free()


def test_score_without_rows_and_repeat():
    """out = lse = NULL: the fused head alone gives the same scores, bit for
    bit, and a repeated call reproduces them (stale partial sums from the
    previous call do not leak)."""
    import torch
    st = workloads.make("qwen3_0p6b")
    case = setup(st)
    a = setup_score(case)
    assert run_score(case, a) == 0
    b = setup_score(case, with_rows=False)
    assert run_score(case, b) == 0
    assert torch.equal(a.score, b.score) and torch.equal(a.logits, b.logits)
    s1 = b.score.clone()
    assert run_score(case, b) == 0
    assert torch.equal(s1, b.score)
    del case, a, b
    _free()
