"""dopr_prefix_attn_noalloc (the entry point for callers that cannot
allocate) against dopr_prefix_attn on the same inputs: two calls in a row on
one device, the second on a smaller batch, then the pass kernel from the
library's scratch.  Every tile shape of the attention gives the same bits,
so the outputs must be bitwise equal to the workspace entry point's.  Size
and argument errors are checked on the host side of the call."""
import ctypes

import numpy as np
import pytest

import workloads
from gpu_harness import compare, log, run, setup

pytestmark = pytest.mark.gpu


def _structure(seed, hq, hkv, lens, n_pairs, t_choices, name):
    rng = np.random.default_rng(seed)
    lens = np.asarray(lens, np.int32)
    doc_ids = rng.integers(0, len(lens), n_pairs).astype(np.int32)
    seqlens = rng.choice(np.asarray(t_choices), n_pairs).astype(np.int32)
    return workloads.custom(lens, doc_ids, seqlens, hq, hkv, name=name)


def _noalloc(case, variant):
    import torch
    import paper_2609_03311_amd as D
    st = case.st
    o, p = case.online, case.prm
    D_ = case.store.head_dim
    out = torch.full((st.n_tokens, st.n_q_heads, D_), float("nan"),
                     dtype=torch.bfloat16, device="cuda")
    lse = torch.full((st.n_tokens, st.n_q_heads), float("nan"),
                     dtype=torch.float32, device="cuda")
    D.dopr_prefix_attn_noalloc(case.store, 0, case.doc_ids, case.cu, o["q"],
                               o["k"], o["v"], p["q_norm_w"], p["k_norm_w"],
                               out, max_tokens=case.step.max_tokens, lse=lse,
                               total_tokens=st.n_tokens,
                               kernel_variant=variant)
    torch.cuda.synchronize()
    assert D.dopr_check_status(case.store) == 0
    return out, lse


def _check_equal(case, out, lse, what):
    import torch
    assert torch.equal(out.view(torch.int16), case.step.out.view(torch.int16)), \
        f"{what}: O differs from dopr_prefix_attn"
    assert torch.equal(lse, case.step.lse), f"{what}: lse differs"


def test_noalloc_matches_workspace_entry_point_twice():
    import gc
    import torch
    # first call: prefixes up to 257 slots (one 8-wave block per CU, long
    # prefixes streamed), ragged T across several 32-row tiles
    big = _structure(300, 16, 8, [0, 1, 15, 16, 17, 31, 32, 33, 63, 64, 65,
                                  255, 256, 257], 40, [1, 2, 17, 33, 129],
                     "noalloc_big")
    # second call, smaller: every prefix within 96 slots (two blocks per CU)
    small = _structure(301, 8, 2, [3, 70, 0], 10, [2, 31, 64, 65],
                       "noalloc_small")
    for st in (big, small):
        log(f"== {st.name} P={st.n_pairs} Ntok={st.n_tokens}")
        case = setup(st, seed=5)
        assert run(case) == 0           # dopr_prefix_attn with a workspace
        out, lse = _noalloc(case, 0)
        _check_equal(case, out, lse, st.name)
        compare(case, np.arange(st.n_pairs))   # and the oracle
        if st is small:
            # the pass kernel, its k^ buffer in the scratch as well
            out8, lse8 = _noalloc(case, 8)
            _check_equal(case, out8, lse8, st.name + " variant 8")
        del case
        gc.collect()
        torch.cuda.empty_cache()


def test_noalloc_rejects_workspace_and_oversized_plans():
    import torch
    import paper_2609_03311_amd as D
    st = _structure(302, 8, 8, [5, 40], 4, [3, 9], "noalloc_err")
    case = setup(st, seed=6)
    L = D.lib()
    o, p = case.online, case.prm
    a = D._attn_args(case.store, case.doc_ids, case.cu, o["q"], o["k"], o["v"],
                     p["q_norm_w"], p["k_norm_w"], case.step.out, None,
                     case.step.workspace, max_tokens=case.step.max_tokens,
                     total_tokens=st.n_tokens)
    assert L.dopr_prefix_attn_noalloc(case.store.handle, 0, ctypes.byref(a),
                                      None) == D.DOPR_ERR_INVALID_ARG
    assert "workspace must be NULL" in D.dopr_last_error()
    # a plan beyond the scratch: the rotary table alone of 2^20 online
    # positions is 512 MiB; rejected on the host before any launch
    a.workspace, a.workspace_bytes = None, 0
    a.max_tokens, a.total_tokens = 1 << 20, 1 << 20
    assert L.dopr_prefix_attn_noalloc(case.store.handle, 0, ctypes.byref(a),
                                      None) == D.DOPR_ERR_WORKSPACE
    assert "no-alloc" in D.dopr_last_error()
    torch.cuda.synchronize()
    assert D.dopr_check_status(case.store) == 0
