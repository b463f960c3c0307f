"""The oracle's pins catch plausible mistakes (CPU).

Each case plants one mistake in a copy of the oracle's C source, builds it
with gcc into a temporary directory and runs the whole pin battery against
it in a subprocess (a planted mistake may crash).  The case passes only if
at least one pin fails.  The real oracle source is never modified.
"""
import os
import subprocess
import sys
import tempfile

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "dopr_oracle.c")

# (id, exact text in the oracle source, replacement)
MUTATIONS = [
    ("rope_sin_sign_first", "x[i] = a * c - b * s;", "x[i] = a * c + b * s;"),
    ("rope_sin_sign_second", "x[i + half] = b * c + a * s;",
     "x[i + half] = b * c - a * s;"),
    ("rope_freq_exponent", "pow(theta, -2.0 * (double)i / (double)d)",
     "pow(theta, -1.0 * (double)i / (double)d)"),
    ("rope_halves_swapped", "double a = x[i], b = x[i + half];",
     "double a = x[i + half], b = x[i];"),
    ("rmsnorm_no_eps", "sqrt(ss / (double)n + eps)", "sqrt(ss / (double)n)"),
    ("rmsnorm_no_weight", "y[i] = w[i] * (x[i] * inv);",
     "y[i] = (x[i] * inv);"),
    ("rmsnorm_sum_not_mean", "sqrt(ss / (double)n + eps)", "sqrt(ss + eps)"),
    ("q_position_not_offset",
     "rope(qhat, D, (double)(L + j), rope_theta, rope_inv_freq);",
     "rope(qhat, D, (double)(j), rope_theta, rope_inv_freq);"),
    ("k_position_not_offset",
     "rope(dst, D, (double)(L + j), rope_theta, rope_inv_freq);",
     "rope(dst, D, (double)(j), rope_theta, rope_inv_freq);"),
    ("rope_ignores_given_freqs", "double freq = inv_freq ? inv_freq[i]",
     "double freq = 0 ? inv_freq[i]"),
    ("q_normed_without_gains",
     "if (qk_norm)\n          rms_norm(x, wq, D, rms_eps, qhat);",
     "if (1)\n          rms_norm(x, wq, D, rms_eps, qhat);"),
    ("k_normed_without_gains",
     "if (qk_norm)\n          rms_norm(x, wk, D, rms_eps, dst);",
     "if (1)\n          rms_norm(x, wk, D, rms_eps, dst);"),
    ("gqa_interleaved", "const int g = h / n_rep;", "const int g = h % Hkv;"),
    ("self_key_dropped", "const int n_keys = L + j + 1;",
     "const int n_keys = L + j;"),
    ("prefix_unscaled", "z[t] = softmax_scale * dot;", "z[t] = dot;"),
    ("own_unscaled", "z[L + t] = softmax_scale * dot;", "z[L + t] = dot;"),
    ("prefix_values_are_keys", "const uint16_t *vt = pv +",
     "const uint16_t *vt = pk +"),
    ("own_values_are_keys", "const double *vt = vown +",
     "const double *vt = khat +"),
    ("lse_without_max", "zmax + log(denom)", "log(denom)"),
    ("q_norm_uses_k_weight", "rms_norm(x, wq, D, rms_eps, qhat);",
     "rms_norm(x, wk, D, rms_eps, qhat);"),
    ("score_sign", "score[p] = ly - ln;", "score[p] = ln - ly;"),
    ("score_rows_indexed_by_token",
     "const int64_t orow = last_only ? p : tok0 + j;",
     "const int64_t orow = tok0 + j;"),
    ("score_rows_first_token", "for (int jq = j0; jq < T; ++jq)",
     "for (int jq = 0; jq < (last_only ? 1 : T); ++jq)"),
    ("score_yes_row_is_no_row", "wy[i] = bf16_to_double(w_head[i]);",
     "wy[i] = bf16_to_double(w_head[width + i]);"),
    ("score_no_norm_weight", "w[i] = bf16_to_double(norm_w[i]);",
     "w[i] = 1.0;"),
    ("group_ptr_shifted", "group_ptr[g] = (int32_t)run;\n      ++g;",
     "group_ptr[g] = (int32_t)(run + c);\n      ++g;"),
    ("store_bytes_k_only", "* n_kv_heads * head_dim * 2 * 2;",
     "* n_kv_heads * head_dim * 2;"),
]

RUNNER = r"""
import sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle, oracle_pins
L = oracle.load_library({lib!r})
order = sorted(oracle_pins.ALL_PINS, key=lambda p: p is oracle_pins.pin_sdpa)
for pin in order:
    try:
        pin(L)
    except Exception as e:
        print("CAUGHT", pin.__name__, type(e).__name__)
        sys.exit(0)
print("MISSED")
"""


@pytest.mark.parametrize("mid,pattern,repl", MUTATIONS,
                         ids=[m[0] for m in MUTATIONS])
def test_pins_catch_planted_mistake(mid, pattern, repl, tmp_path):
    src = open(SRC).read()
    assert src.count(pattern) == 1, f"{mid}: pattern must occur exactly once"
    mutated = tmp_path / "mutated.c"
    mutated.write_text(src.replace(pattern, repl))
    lib = str(tmp_path / "libmutated.so")
    oracle.build(str(mutated), lib)
    code = RUNNER.format(root=ROOT, tests=os.path.dirname(__file__), lib=lib)
    r = subprocess.run([sys.executable, "-c", code], capture_output=True,
                       text=True, timeout=300)
    out = r.stdout + r.stderr
    assert "MISSED" not in r.stdout, f"{mid}: no pin failed\n{out[-2000:]}"
    # a crash (nonzero exit without CAUGHT) also counts as caught
    assert "CAUGHT" in r.stdout or r.returncode != 0, out[-2000:]


# Mistakes planted in the Python decoder-layer oracle (oracle/__init__.py):
# the pin battery runs against a copy of that module with one change.
PY_SRC = os.path.join(ROOT, "oracle", "__init__.py")
PY_MUTATIONS = [
    ("layer_attn_residual_dropped", "x2 = X + att.reshape", "x2 = att.reshape"),
    ("layer_mlp_residual_dropped", "y = x2 + a @", "y = a @"),
    ("layer_silu_missing", "a = g / (1.0 + np.exp(-g)) * u", "a = g * u"),
    ("layer_gate_is_up", 'g = h2 @ w["w_gate"].T', 'g = h2 @ w["w_up"].T'),
    ("layer_norm_gain_missing", "return w * (x / np.sqrt(",
     "return (x / np.sqrt("),
    ("layer_mlp_norm_is_attn_norm", 'h2 = _rms_norm_rows(x2, w["mlp_norm"]',
     'h2 = _rms_norm_rows(x2, w["attn_norm"]'),
]

PY_RUNNER = r"""
import importlib.util, sys
sys.path[:0] = [{root!r}, {tests!r}]
import oracle as real
spec = importlib.util.spec_from_file_location("oracle_mut", {path!r})
mut = importlib.util.module_from_spec(spec)
spec.loader.exec_module(mut)
mut._lib = real.lib()
import oracle_pins
oracle_pins.oracle = mut
try:
    oracle_pins.pin_decoder_layer(real.lib())
except Exception as e:
    print("CAUGHT", type(e).__name__)
    sys.exit(0)
print("MISSED")
"""


@pytest.mark.parametrize("mid,pattern,repl", PY_MUTATIONS,
                         ids=[m[0] for m in PY_MUTATIONS])
def test_pins_catch_planted_layer_mistake(mid, pattern, repl, tmp_path):
    src = open(PY_SRC).read()
    assert src.count(pattern) == 1, f"{mid}: pattern must occur exactly once"
    mutated = tmp_path / "oracle_mut.py"
    mutated.write_text(src.replace(pattern, repl))
    code = PY_RUNNER.format(root=ROOT, tests=os.path.dirname(__file__),
                            path=str(mutated))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True,
                       text=True, timeout=300)
    out = r.stdout + r.stderr
    assert "MISSED" not in r.stdout, f"{mid}: no pin failed\n{out[-2000:]}"
    assert "CAUGHT" in r.stdout or r.returncode != 0, out[-2000:]
