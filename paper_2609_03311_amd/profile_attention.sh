#!/bin/bash
# Collect the rocprofv3 summaries of one workload's attention launches:
#   <tag>_<config>_kernel_stats.txt  per-kernel durations (--kernel-trace --stats)
#   <tag>_<config>_traffic.txt       HBM bytes per step (FETCH_SIZE, WRITE_SIZE,
#                                    each scaled by a 1 GiB copy kernel)
#   <tag>_<config>_pmc.txt           MFMA / VALU / LDS utilisation and waits
# tag: k_pass_attn (full layer: k^ precompute + pass kernel) or k_score_rows
# (last-layer scoring).  Raw output stays in gpurun_out/prof_<path>_<config>/;
# the summaries are written to gpurun_out/summaries/.
# usage: bash paper_2609_03311_amd/profile_attention.sh CONFIG full|score [D]
#        [summarize]   (the last form only rewrites the summaries from the
#                       raw output already in gpurun_out/prof_<path>_<config>/)
set -o pipefail
cfg=$1
path=$2
D=${3:-128}
only_summarize=$4
R=$(cd "$(dirname "$0")/.." && pwd)
out=$R/gpurun_out/prof_${path}_${cfg}
sum=$R/gpurun_out/summaries
mkdir -p "$out" "$sum"
if [ "$path" = score ]; then
  tag=k_score_rows
  kern="k_score_rows<$D>"
else
  tag=k_pass_attn
  kern="k_own_khat<$D>|k_pass_attn<$D>"
fi
args="--config $cfg --path $path --steps 3 --warmup 1 --no-cpu-baseline"
bench="python3 bench.py $args"   # as recorded (run from the repository root)
me="bash paper_2609_03311_amd/profile_attention.sh $cfg $path $D"
cd /tmp && export TMPDIR=/tmp

step() {  # name, extra bench options, rocprofv3 options...
  local name=$1 extra=$2
  shift 2
  echo "== $name" && timeout -k 10 -s KILL 240 rocprofv3 "$@" -d "$out/$name" \
    -o run --output-format csv -- python3 "$R/bench.py" $args $extra \
    > "$out/$name.log" 2>&1
  local rc=$?
  tail -1 "$out/$name.log" | cut -c1-160
  return $rc
}

if [ "$only_summarize" != summarize ]; then
  step stats "" --kernel-trace --stats &&
    step fetch --copy-calibration --pmc FETCH_SIZE &&
    step write --copy-calibration --pmc WRITE_SIZE &&
    step pmc_a "" --pmc $(python3 -c "import sys; sys.path.insert(0, '$R'); from paper_2609_03311_amd import profiling as p; print(p.PMC_PASSES[0])") &&
    step pmc_b "" --pmc $(python3 -c "import sys; sys.path.insert(0, '$R'); from paper_2609_03311_amd import profiling as p; print(p.PMC_PASSES[1])") ||
    exit $?
fi

cd "$R" &&
  python3 -m paper_2609_03311_amd.profiling stats "$out/stats" \
    --command "$me (rocprofv3 --kernel-trace --stats -- $bench)" \
    > "$sum/${tag}_${cfg}_kernel_stats.txt" &&
  python3 -m paper_2609_03311_amd.profiling traffic "$out/fetch" "$out/write" \
    --kernel "$kern" \
    --command "$me (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE -- $bench --copy-calibration)" \
    > "$sum/${tag}_${cfg}_traffic.txt" &&
  python3 -m paper_2609_03311_amd.profiling pmc "$out/pmc_a" "$out/pmc_b" \
    --kernel "$kern" \
    --command "$me (rocprofv3 --pmc <PMC_PASSES[0]>, then <PMC_PASSES[1]> -- $bench)" \
    > "$sum/${tag}_${cfg}_pmc.txt"
