"""The C ABI on the CPU: the library loads, exports every function the header
declares, the Python binding's struct layouts equal the C ones, and
host-side validation returns the documented status codes without touching a
GPU."""
import ctypes
import os
import re
import subprocess

import numpy as np
import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dopr.h")


def _D():
    import paper_2609_03311_amd as D
    D.lib()
    return D


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dopr_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_function():
    D = _D()
    names = header_functions()
    assert len(names) >= 12
    L = ctypes.CDLL(D.LIB_PATH)
    for n in names:
        assert hasattr(L, n), f"{n} not exported"
    assert set(names) == set(D.EXPORTS), "binding and header disagree"


def test_struct_layouts_match_header(tmp_path):
    D = _D()
    probe = tmp_path / "probe.c"
    structs = {"dopr_store_desc_t": D._StoreDesc,
               "dopr_attn_args_t": D._AttnArgs,
               "dopr_score_args_t": D._ScoreArgs,
               "dopr_score_head_t": D._ScoreHead,
               "dopr_layer_args_t": D._LayerArgs,
               "dopr_salience_args_t": D._SalienceArgs}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "dopr.h"',
             "int main(void) {"]
    for cname, py in structs.items():
        lines.append(f'printf("{cname} size %zu\\n", sizeof({cname}));')
        for f, _ in py._fields_:
            lines.append(f'printf("{cname} {f} %zu\\n", '
                         f'offsetof({cname}, {f}));')
    lines += ["return 0; }"]
    probe.write_text("\n".join(lines))
    exe = tmp_path / "probe"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"),
                    str(probe), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True,
                         check=True).stdout.split("\n")
    got = {}
    for line in out:
        if line:
            s, f, v = line.split()
            got[(s, f)] = int(v)
    for cname, py in structs.items():
        assert got[(cname, "size")] == ctypes.sizeof(py), cname
        for f, _ in py._fields_:
            assert got[(cname, f)] == getattr(py, f).offset, (cname, f)


def test_store_bytes_closed_form():
    D = _D()
    rng = np.random.default_rng(0)
    for layers, hkv in [(1, 8), (36, 8), (28, 8), (3, 2)]:
        doc_len = rng.integers(-1, 300, 500).astype(np.int32)
        pool, payload = D.dopr_store_bytes(layers, hkv, 128, doc_len)
        assert payload == oracle.store_payload_bytes(layers, hkv, 128,
                                                     doc_len)
        # index (12 B/doc), key-norm bounds (4 B per doc, layer and kv
        # head) and the payload with V rows padded to 8 slots
        res = doc_len[doc_len >= 0].astype(np.int64)
        padded = ((res + 7) // 8 * 8 + res).sum() * layers * hkv * 128 * 2
        index = (12 + 4 * layers * hkv) * len(doc_len)
        assert pool >= padded + index
        assert pool <= padded + index + 4 * 256 + 256


def test_host_validation_codes():
    D = _D()
    for bad_d in (96, 32, 256):
        with pytest.raises(D.DoprError) as e:
            D.dopr_store_bytes(1, 8, bad_d, [4])
        assert e.value.status == D.DOPR_ERR_UNSUPPORTED
    # head size 64 (Llama 3.2 1B) is laid out like 128, at half the bytes
    _, p64 = D.dopr_store_bytes(2, 8, 64, [4, 0, 13])
    _, p128 = D.dopr_store_bytes(2, 8, 128, [4, 0, 13])
    assert p64 == oracle.store_payload_bytes(2, 8, 64, np.array([4, 0, 13]))
    assert 2 * p64 == p128
    with pytest.raises(D.DoprError) as e:
        D.dopr_store_bytes(1, 8, 128, [4, -2])
    assert e.value.status == D.DOPR_ERR_INVALID_ARG
    with pytest.raises(D.DoprError) as e:
        D.dopr_store_bytes(0, 8, 128, [4])
    assert e.value.status == D.DOPR_ERR_INVALID_ARG
    L = D.lib()
    a = D._AttnArgs()
    n = ctypes.c_size_t(0)
    assert L.dopr_prefix_attn_workspace(None, ctypes.byref(a),
                                        ctypes.byref(n)) == \
        D.DOPR_ERR_INVALID_ARG
    assert "store is NULL" in D.dopr_last_error()
    assert L.dopr_prefix_attn(None, 0, ctypes.byref(a), None) == \
        D.DOPR_ERR_INVALID_ARG
    s = D._ScoreArgs()
    s.n_pairs, s.width, s.h_row_stride, s.rms_eps = 4, 12, 12, 1e-6
    assert L.dopr_score_logits(ctypes.byref(s), None) == \
        D.DOPR_ERR_INVALID_ARG
    s.width, s.h_row_stride = 16, 8
    assert L.dopr_score_logits(ctypes.byref(s), None) == \
        D.DOPR_ERR_INVALID_ARG
    s.h_row_stride = 16
    assert L.dopr_score_logits(ctypes.byref(s), None) == \
        D.DOPR_ERR_INVALID_ARG  # NULL buffers
    s.n_pairs = 0
    assert L.dopr_score_logits(ctypes.byref(s), None) == D.DOPR_OK
    hd = D._ScoreHead()
    assert L.dopr_prefix_attn_score(None, 0, ctypes.byref(a), None, None) == \
        D.DOPR_ERR_INVALID_ARG
    assert "head is NULL" in D.dopr_last_error()
    assert L.dopr_prefix_attn_score(None, 0, ctypes.byref(a),
                                    ctypes.byref(hd), None) == \
        D.DOPR_ERR_INVALID_ARG
    assert "store is NULL" in D.dopr_last_error()
    assert L.dopr_prefix_attn_score_workspace(None, ctypes.byref(a),
                                              ctypes.byref(n)) == \
        D.DOPR_ERR_INVALID_ARG
    la = D._LayerArgs()
    assert L.dopr_decoder_layer(None, 0, ctypes.byref(a), ctypes.byref(la),
                                None) == D.DOPR_ERR_INVALID_ARG
    assert L.dopr_decoder_layer_workspace(None, ctypes.byref(a),
                                          ctypes.byref(la),
                                          ctypes.byref(n)) == \
        D.DOPR_ERR_INVALID_ARG
    assert L.dopr_check_status(None, None) == D.DOPR_ERR_INVALID_ARG
    assert D.dopr_status_str(D.DOPR_ERR_DOC_RANGE) == "DOPR_ERR_DOC_RANGE"
    assert D.dopr_status_str(D.DOPR_ERR_SEQLEN) == "DOPR_ERR_SEQLEN"
    assert L.dopr_store_destroy(None) == D.DOPR_OK


def test_salience_host_validation_and_workspace():
    """Salience argument checks and workspace sizes (host arithmetic only):
    the row log-sum-exp of every (token, q head), the largest key norm of
    every (document, kv head), plus the head-averaged matrix of as many
    documents as fit in 1 GiB unless the caller keeps it."""
    D = _D()
    L = D.lib()

    def up(n):
        return -(-n // 256) * 256

    ws = D.dopr_salience_workspace(n_docs=64, max_doclen=2048, n_q_heads=32,
                                   n_kv_heads=8, top_p=8,
                                   total_tokens=64 * 2048)
    lse = 4 * 32 * 64 * 2048
    kn = up(4 * 8 * 64 * 8)               # 8 partial maxima per doc, head
    assert ws == lse + kn + (1 << 30)     # 64 docs of 16 MiB in one pass
    ws = D.dopr_salience_workspace(n_docs=3, max_doclen=2048, n_q_heads=32,
                                   n_kv_heads=8, top_p=8, total_tokens=5000)
    assert ws == up(4 * 32 * 5000) + up(4 * 8 * 3 * 8) + 3 * 2048 * 2048 * 4
    ws = D.dopr_salience_workspace(n_docs=3, max_doclen=2048, n_q_heads=32,
                                   n_kv_heads=8, top_p=8, total_tokens=5000,
                                   with_attention=True)
    assert ws == up(4 * 32 * 5000) + up(4 * 8 * 3 * 8)
    assert D.dopr_salience_workspace(n_docs=0, max_doclen=5, n_q_heads=2,
                                     n_kv_heads=1, top_p=1,
                                     total_tokens=0) == 0
    bad = [dict(max_doclen=4097, code=D.DOPR_ERR_UNSUPPORTED),
           dict(max_doclen=0, code=D.DOPR_ERR_INVALID_ARG),
           dict(top_p=65, code=D.DOPR_ERR_UNSUPPORTED),
           dict(top_p=0, code=D.DOPR_ERR_INVALID_ARG),
           dict(n_q_heads=12, n_kv_heads=8, code=D.DOPR_ERR_INVALID_ARG),
           dict(n_docs=-1, code=D.DOPR_ERR_INVALID_ARG)]
    for b in bad:
        kw = dict(n_docs=2, max_doclen=64, n_q_heads=16, n_kv_heads=8,
                  top_p=8, total_tokens=100)
        code = b.pop("code")
        kw.update(b)
        with pytest.raises(D.DoprError) as e:
            D.dopr_salience_workspace(**kw)
        assert e.value.status == code, b
    a = D._SalienceArgs()
    a.n_docs, a.max_doclen, a.n_q_heads, a.n_kv_heads = 2, 64, 16, 8
    a.top_p, a.softmax_scale, a.total_tokens = 8, 0.088, 100
    assert L.dopr_salience(ctypes.byref(a), None) == D.DOPR_ERR_INVALID_ARG
    assert "cu_doclens and u" in D.dopr_last_error()
    a.cu_doclens, a.u = 256, 256          # never dereferenced on the host
    assert L.dopr_salience(ctypes.byref(a), None) == D.DOPR_ERR_INVALID_ARG
    assert "q and k" in D.dopr_last_error()
    a.q, a.k = 256, 256
    assert L.dopr_salience(ctypes.byref(a), None) == D.DOPR_ERR_WORKSPACE
    # the row pass relies on a positive scale (the chunk maximum stays the
    # largest scaled logit): zero, negative and non-finite scales are refused
    for bad in (0.0, -0.088, float("inf"), float("nan")):
        a.softmax_scale = bad
        assert L.dopr_salience(ctypes.byref(a), None) == \
            D.DOPR_ERR_INVALID_ARG, bad
        assert "softmax_scale" in D.dopr_last_error()
        n = ctypes.c_size_t(0)
        assert L.dopr_salience_workspace(ctypes.byref(a), ctypes.byref(n)) \
            == D.DOPR_ERR_INVALID_ARG, bad
    a.softmax_scale = 0.088
    a.selected = 256
    assert L.dopr_select_top_k(ctypes.byref(a), None) == \
        D.DOPR_ERR_INVALID_ARG
    assert "cu_select" in D.dopr_last_error()
    a.n_docs = 0
    assert L.dopr_select_top_k(ctypes.byref(a), None) == D.DOPR_OK
