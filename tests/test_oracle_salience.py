"""The salience oracle (Sec. 3.2.1) against its pins, and the pins against
plausible mistakes planted in a copy of the oracle (CPU)."""
import os
import subprocess
import sys

import pytest

import salience_pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "salience.py")


@pytest.mark.parametrize("pin", salience_pins.ALL_PINS,
                         ids=[p.__name__ for p in salience_pins.ALL_PINS])
def test_salience_pin(pin):
    pin()


# (id, exact text in oracle/salience.py, replacement)
MUTATIONS = [
    ("mean_over_kv_heads", "return total / Hq", "return total / Hkv"),
    ("gqa_interleaved", "k[:, h // n_rep, :]", "k[:, h % Hkv, :]"),
    ("no_causal_mask", "z = np.where(visible, z, -np.inf)", "z = z"),
    ("no_softmax_scale", "z = softmax_scale * (q[:, h, :]", "z = (q[:, h, :]"),
    ("tp_counts_masked_entry", "m = min(p, n - i)", "m = min(p, n - i + 1)"),
    ("tp_divides_by_p", "u[i] = largest.sum() / m", "u[i] = largest.sum() / p"),
    ("row_not_column", "column = abar[i:, i]", "column = abar[i, :i + 1]"),
    ("smallest_not_largest", "np.sort(column)[::-1][:m]",
     "np.sort(column)[:m]"),
    ("ties_to_higher_position", "key=lambda i: (-u[i], i)",
     "key=lambda i: (-u[i], -i)"),
    ("rank_order_output", "np.array(sorted(ranked[:k])",
     "np.array((ranked[:k])"),
    ("bf16_shift", "<< 16).view(np.float32)", "<< 15).view(np.float32)"),
]

RUNNER = r"""
import importlib.util, sys
sys.path[:0] = [{root!r}, {tests!r}]
spec = importlib.util.spec_from_file_location("salience_mut", {path!r})
mut = importlib.util.module_from_spec(spec)
spec.loader.exec_module(mut)
import salience_pins
salience_pins.salience = mut
for pin in salience_pins.ALL_PINS:
    try:
        pin()
    except Exception as e:
        print("CAUGHT", pin.__name__, type(e).__name__)
        sys.exit(0)
print("MISSED")
"""


@pytest.mark.parametrize("mid,pattern,repl", MUTATIONS,
                         ids=[m[0] for m in MUTATIONS])
def test_pins_catch_planted_salience_mistake(mid, pattern, repl, tmp_path):
    src = open(SRC).read()
    assert src.count(pattern) == 1, f"{mid}: pattern must occur exactly once"
    mutated = tmp_path / "salience_mut.py"
    mutated.write_text(src.replace(pattern, repl))
    code = RUNNER.format(root=ROOT, tests=os.path.dirname(__file__),
                         path=str(mutated))
    r = subprocess.run([sys.executable, "-c", code], capture_output=True,
                       text=True, timeout=300)
    out = r.stdout + r.stderr
    assert "MISSED" not in r.stdout, f"{mid}: no pin failed\n{out[-2000:]}"
    assert "CAUGHT" in r.stdout or r.returncode != 0, out[-2000:]
