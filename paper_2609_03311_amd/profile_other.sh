#!/bin/bash
# Collect the rocprofv3 summaries of the paths other than attention:
#   salience_qwen3_8b_docs_kernel_stats.txt, salience_qwen3_8b_docs_pmc.txt
#       offline salience selection (row LSE and mean-attention kernels)
#   decoder_layer_<config>_kernel_stats.txt   one decoder layer (Qwen3-0.6B
#       and Qwen3-8B shapes)
#   store_ingest_qwen3_8b_kernel_stats.txt    prefix-store ingest
# Raw output stays in gpurun_out/prof_other/; the summaries are written to
# gpurun_out/summaries/.
# usage: bash paper_2609_03311_amd/profile_other.sh [summarize]
set -o pipefail
only_summarize=$1
R=$(cd "$(dirname "$0")/.." && pwd)
out=$R/gpurun_out/prof_other
sum=$R/gpurun_out/summaries
mkdir -p "$out" "$sum"
me="bash paper_2609_03311_amd/profile_other.sh"
sal="--path salience --config qwen3_8b_docs --steps 5 --warmup 1 --no-cpu-baseline"
lay="--path layer --steps 5 --warmup 2 --no-cpu-baseline"
ing="--path ingest --steps 5 --warmup 1"
pm() { python3 -c "import sys; sys.path.insert(0, '$R'); from paper_2609_03311_amd import profiling as p; print(p.PMC_PASSES[$1])"; }
cd /tmp && export TMPDIR=/tmp

step() {  # name, bench options (one word-split string), rocprofv3 options...
  local name=$1 opts=$2
  shift 2
  echo "== $name" && timeout -k 10 -s KILL 300 rocprofv3 "$@" -d "$out/$name" \
    -o run --output-format csv -- python3 "$R/bench.py" $opts \
    > "$out/$name.log" 2>&1
  local rc=$?
  tail -1 "$out/$name.log" | cut -c1-160
  return $rc
}

if [ "$only_summarize" != summarize ]; then
  step sal_stats "$sal" --kernel-trace --stats &&
    step sal_pmc_a "$sal" --pmc $(pm 0) &&
    step sal_pmc_b "$sal" --pmc $(pm 1) &&
    step layer_qwen3_0p6b "$lay --config qwen3_0p6b" --kernel-trace --stats &&
    step layer_qwen3_8b "$lay --config qwen3_8b" --kernel-trace --stats &&
    step ingest "$ing" --kernel-trace --stats ||
    exit $?
fi

P="python3 -m paper_2609_03311_amd.profiling"
cd "$R" &&
  $P stats "$out/sal_stats" --sources salience \
    --command "$me (rocprofv3 --kernel-trace --stats -- python3 bench.py $sal)" \
    > "$sum/salience_qwen3_8b_docs_kernel_stats.txt" &&
  $P pmc "$out/sal_pmc_a" "$out/sal_pmc_b" --sources salience \
    --kernel "k_row_lse<|k_mean_attn" \
    --command "$me (rocprofv3 --pmc <PMC_PASSES[0]>, then <PMC_PASSES[1]> -- python3 bench.py $sal)" \
    > "$sum/salience_qwen3_8b_docs_pmc.txt" &&
  for c in qwen3_0p6b qwen3_8b; do
    $P stats "$out/layer_$c" --sources layer \
      --command "$me (rocprofv3 --kernel-trace --stats -- python3 bench.py $lay --config $c)" \
      > "$sum/decoder_layer_${c}_kernel_stats.txt" || exit $?
  done &&
  $P stats "$out/ingest" --sources store \
    --command "$me (rocprofv3 --kernel-trace --stats -- python3 bench.py $ing)" \
    > "$sum/store_ingest_qwen3_8b_kernel_stats.txt"
