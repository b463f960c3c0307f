"""Host-side checks of the measurement tooling (CPU): the source hashes the
profile summaries carry, the bench table, the bench's use of a committed
summary, and the pass-kernel phase summary."""
import json
import os

import numpy as np

import bench
from paper_2609_03311_amd import phase_timing, profiling


def test_source_hash_ignores_comments_and_layout(tmp_path, monkeypatch):
    a = "int f(int x) {\n  return x + 1;  // one\n}\n/* block */\n"
    b = "int f(int x)   {   return x + 1; }\n// another comment\n"
    c = "int f(int x) { return x + 2; }\n"
    assert profiling._code_only(a) == profiling._code_only(b)
    assert profiling._code_only(a) != profiling._code_only(c)
    # every kind names sources that exist, and the kinds hash differently
    shas = {k: profiling.kernel_source_sha(k) for k in profiling.SOURCE_SETS}
    assert len(set(shas.values())) == len(shas)
    for k, srcs in profiling.SOURCE_SETS.items():
        for rel in srcs:
            assert os.path.exists(os.path.join(profiling.HERE, rel)), rel
    # the attention kind's summary line is the one the bench matches
    assert profiling._sha_lines("attention") == [
        f"kernel_source_sha: {shas['attention']}"]
    assert profiling._sha_lines("salience")[1].startswith("kernel_sources: ")


def test_bench_table_rows(tmp_path):
    line = {"metric": "m", "value": 1234.5, "unit": "pairs/s",
            "ms_per_step": 2.5, "attention_ms": 2.0,
            "config": {"name": "qwen3_8b", "path": "full online layer",
                       "queue_order": 0},
            "roofline": {"achieved": 4000.0, "unit": "GB/s", "frac": 0.5,
                         "traffic": 90e9},
            "mfma_util": 0.25}
    p = tmp_path / "a.jsonl"
    p.write_text(json.dumps(line) + "\n")
    out = profiling.bench_table([str(p)], "cmd")
    row = [r for r in out.splitlines() if r.startswith("qwen3_8b")]
    assert len(row) == 1
    assert "4000.0" in row[0] and "0.5000" in row[0]
    assert "90.00" in row[0] and "0.250" in row[0]


def test_phase_summary_shares():
    t = np.zeros((8, phase_timing.N_SLOTS))
    rng = np.random.default_rng(0)
    t[:, :len(phase_timing.PHASES)] = rng.integers(
        1, 1000, (8, len(phase_timing.PHASES)))
    t[:, phase_timing.UNITS] = 10
    t[:, phase_timing.PASSES] = 43
    t[:, phase_timing.TAILS] = 8
    t[:, phase_timing.TAIL_CYC] = 100
    s = phase_timing.summary("qwen3_8b", 5, t, 34.5, "cmd")
    rows = [r for r in s.splitlines()
            if any(r.startswith(n) for n in phase_timing.PHASES)]
    assert len(rows) == len(phase_timing.PHASES)
    # each wave's shares add up to 100 %
    shares = np.array([[float(x.rstrip("%")) for x in r[26:].split()]
                       for r in rows])
    assert np.allclose(shares[:, :8].sum(axis=0), 100.0, atol=0.05)
    assert "4.30 per unit" in s and "8 per step" not in s
    assert "passes of at most 32 rows: 2 per step" in s


def test_bench_reads_only_matching_summaries(tmp_path, monkeypatch):
    """A committed summary counts only while its source hash matches the
    current sources and the run used the default kernel; a stale one
    yields no traffic figure."""
    prof = tmp_path / "profiles"
    prof.mkdir()
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    (prof / "k_pass_attn_qwen3_8b_traffic.txt").write_text(
        f"kernel_source_sha: {profiling.kernel_source_sha()}\n"
        "traffic_bytes_per_launch: 123\n")
    (prof / "k_pass_attn_llama3_2_1b_traffic.txt").write_text(
        "kernel_source_sha: 0000000000000000\n"
        "traffic_bytes_per_launch: 123\n")
    assert bench.measured_traffic("qwen3_8b", 0) == 123
    assert bench.measured_traffic("qwen3_8b", 8) is None    # not default
    assert bench.measured_traffic("llama3_2_1b", 0) is None  # stale
    assert bench.measured_traffic("qwen3_4b", 0) is None     # none
