"""Head size 64 on the GPU vs the float64 oracle: the attention kernels at
D = 64 (the head size of Llama-3.2-1B, the model of the paper's
cross-family check, Appendix "Generalization Across Model Families"), with
QK-norm gains as well as without, in every tile shape, with prefixes longer
than the LDS-resident segment, and the store's put/gather at D = 64.

At D = 64 a 32-key chunk block is 4 KB, so the one-block-per-CU shape keeps
512 prefix slots resident (16 chunks) and the two-blocks-per-CU shape 256
(8 chunks); the 700- and 513-slot prefixes below are streamed in segments
by every shape.  Tolerance: max-abs 2e-2 on O, LSE, logits and score, as at
D = 128 (bf16 operands, fp32 accumulation over half as many products).
Integer work (store put/gather) is compared bit for bit.
"""
import gc

import numpy as np
import pytest

import workloads
from gpu_harness import (compare, log, oracle_subset, run, run_score, setup,
                         setup_score)

pytestmark = pytest.mark.gpu

D = 64
TOL = 2e-2


def _free():
    import torch
    gc.collect()
    torch.cuda.empty_cache()


def _structure(seed, lens, n_pairs, t_choices, name, hq=32, hkv=8):
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens, np.int32)
    doc_ids = rng.integers(0, len(lens), n_pairs).astype(np.int32)
    seqlens = rng.choice(np.asarray(t_choices), n_pairs).astype(np.int32)
    return workloads.custom(lens, doc_ids, seqlens, hq, hkv, name=name,
                            head_dim=D)


# prefixes 0..256 (resident in every shape), T from 1 (score token only) to
# 70 (several own-key chunks)
RAGGED = dict(lens=[256, 0, 33, 100, 7, 192, 65, 1], n_pairs=24,
              t_choices=[1, 2, 31, 33, 70])
# prefixes past the 512 slots the one-block-per-CU shape keeps resident
LONG = dict(lens=[700, 513, 64], n_pairs=10, t_choices=[1, 17, 40])


@pytest.mark.parametrize("variant", [0, 1, 2, 3, 4, 5, 6, 8])
def test_ragged_all_shapes(variant):
    """QK-norm at D = 64, every tile shape (0 automatic, 4 exact mode, 5
    self-check: every unit recomputed exactly), all rows vs the oracle."""
    st = _structure(3, name="d64_ragged", **RAGGED)
    case = setup(st, seed=3, kernel_variant=variant)
    assert run(case) == 0
    compare(case, np.arange(st.n_pairs))
    del case
    _free()


@pytest.mark.parametrize("variant", [0, 1, 6, 8])
def test_long_prefix_segments(variant):
    st = _structure(4, name="d64_long", **LONG)
    case = setup(st, seed=4, kernel_variant=variant)
    assert run(case) == 0
    compare(case, np.arange(st.n_pairs))
    del case
    _free()


def test_gqa_ratios():
    """Other q/kv head ratios at D = 64 (n_rep 1 and 4)."""
    for hq, hkv in ((8, 8), (16, 4)):
        st = _structure(5, name=f"d64_{hq}q{hkv}kv", hq=hq, hkv=hkv,
                        **RAGGED)
        case = setup(st, seed=5)
        assert run(case) == 0
        compare(case, np.arange(st.n_pairs))
        del case
        _free()


def test_score_rows_and_head():
    """Last-layer scoring at D = 64: score-token rows and the fused score
    head (input width Hq * 64) vs the oracle."""
    st = _structure(6, name="d64_score", **RAGGED)
    case = setup(st, seed=6)
    sstep = setup_score(case)
    assert run_score(case, sstep) == 0
    pairs = np.arange(st.n_pairs)
    ref = oracle_subset(case, pairs, last_only=True)
    got = sstep.out.float().cpu().numpy()
    e = float(np.abs(got - ref["out"]).max())
    el = float(np.abs(sstep.lse.cpu().numpy() - ref["lse"]).max())
    es = float(np.abs(sstep.score.cpu().numpy() - ref["score"]).max())
    eg = float(np.abs(sstep.logits.cpu().numpy() - ref["logits"]).max())
    log(f"d64 score: max|dO|={e:.3e} max|dlse|={el:.3e} max|ds|={es:.3e} "
        f"max|dlogit|={eg:.3e}")
    assert (ref["status"] == 0).all()
    assert e <= TOL and el <= TOL and es <= TOL and eg <= TOL
    del case
    _free()


def test_llama3_2_1b_shaped_batch_sampled():
    """The Llama-3.2-1B-shaped batch (20k docs x 256 slots, 25.6k pairs,
    T = 129) at full size in the benchmark's launch configuration, compared
    on sampled pairs (with QK-norm gains; the no-norm rows are covered on
    the Llama-family cases)."""
    st = workloads.make("llama3_2_1b")
    case = setup(st, seed=0)
    assert run(case) == 0
    from gpu_harness import sample_pairs
    compare(case, sample_pairs(st, 24))
    del case
    _free()


def test_store_put_gather_bit_exact():
    """Store layout at D = 64: put then gather returns the canonical states
    bit for bit (ragged lengths incl. 0 and a non-multiple of 8)."""
    import torch
    from paper_2609_03311_amd import (dopr_check_status, dopr_gather_prefix,
                                      pipeline)
    lens = np.array([37, 0, 256, 5, 64, -1, 130], np.int32)
    st = workloads.custom(lens, [0], [1], 32, 8, name="d64_store",
                          head_dim=D)
    k, v, doc_off, _ = workloads.prefix_source(st, "cuda", 9)
    assert k.shape[-1] == D
    store = pipeline.make_store(st.doc_len, 8, k, v)
    want = np.array([6, 2, 0, 4, 3, 2, 1], np.int32)
    cu = np.zeros(len(want) + 1, np.int64)
    np.cumsum(lens[want], out=cu[1:])
    ko = torch.empty((int(cu[-1]), 8, D), dtype=torch.bfloat16,
                     device="cuda")
    vo = torch.empty_like(ko)
    dopr_gather_prefix(store, 0, torch.from_numpy(want).cuda(),
                       torch.from_numpy(cu).cuda(), ko, vo)
    torch.cuda.synchronize()
    assert dopr_check_status(store) == 0
    idx = np.concatenate([np.arange(doc_off[d], doc_off[d] + lens[d])
                          for d in want])
    it = torch.from_numpy(idx).cuda()
    assert torch.equal(ko.view(torch.int16),
                       k.index_select(0, it).view(torch.int16))
    assert torch.equal(vo.view(torch.int16),
                       v.index_select(0, it).view(torch.int16))
