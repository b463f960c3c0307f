#!/bin/bash
# Run bench.py on every workload and path and condense the JSON lines into
# one table (profiles/bench_all_workloads.txt is this script's output).
#   part "attn":   full layer and last-layer scoring on every workload, and
#                  the full layer with the work queues in natural order (1)
#                  against the automatic order (0) on the workloads where the
#                  order matters
#   part "other":  decoder layer, salience selection and store ingest
# Raw JSON lines go to gpurun_out/bench_all/; the table to stdout.
# usage: bash paper_2609_03311_amd/bench_all_workloads.sh attn|other|table
set -o pipefail
R=$(cd "$(dirname "$0")/.." && pwd)
out=$R/gpurun_out/bench_all
mkdir -p "$out"
cd "$R" || exit 1

run() {  # name, bench options...
  local name=$1
  shift
  echo "== $name" >&2
  timeout -k 10 300 python3 -u bench.py "$@" > "$out/$name.log" 2>&1
  local rc=$?
  [ $rc -ne 0 ] && { tail -5 "$out/$name.log" >&2; return $rc; }
  tail -1 "$out/$name.log" >> "$out/$part.jsonl"
}

part=$1
case "$part" in
attn)
  rm -f "$out/attn.jsonl"
  for path in full score; do
    for c in tiny qwen3_0p6b qwen3_4b qwen3_8b qwen3_8b_ragged \
             qwen3_8b_ragged_x8 llama3_8b llama3_2_1b; do
      run "${path}_$c" --config $c --path $path --no-cpu-baseline || exit $?
    done
  done
  for c in qwen3_4b qwen3_0p6b qwen3_8b_ragged qwen3_8b; do
    run "natural_$c" --config $c --queue-order 1 --no-cpu-baseline || exit $?
  done
  ;;
other)
  rm -f "$out/other.jsonl"
  for c in qwen3_0p6b qwen3_4b qwen3_8b; do
    run "layer_$c" --config $c --path layer --steps 5 --warmup 2 \
      --no-cpu-baseline || exit $?
  done
  for c in qwen3_0p6b_docs qwen3_4b_docs qwen3_8b_docs; do
    run "salience_$c" --config $c --path salience --cpu-seconds 10 || exit $?
  done
  echo "== ingest" >&2
  timeout -k 10 300 python3 -u bench.py --path ingest --steps 5 --warmup 1 \
    > "$out/ingest.log" 2>&1 || { tail -5 "$out/ingest.log" >&2; exit 1; }
  grep '^{' "$out/ingest.log" >> "$out/other.jsonl"
  ;;
table)
  python3 -m paper_2609_03311_amd.profiling benchtable \
    "$out/attn.jsonl" "$out/other.jsonl" \
    --command "bash paper_2609_03311_amd/bench_all_workloads.sh attn, then other (bench.py --config/--path/--queue-order per row; layer --steps 5 --warmup 2; salience --cpu-seconds 10; ingest --steps 5 --warmup 1)"
  ;;
*)
  echo "usage: $0 attn|other|table" >&2
  exit 2
  ;;
esac
