#!/bin/bash
# Kernel-trace profile of the benchmark's planning loop (score, top-k, then
# commit-and-advance, repeated): per-kernel durations of the three commit
# kernels next to the scoring kernels.  Raw output under
# gpurun_out/prof_commit_<workload>/; prints the summary.
#   usage: paper_2605_07238_amd/profile_commit.sh <workload> [planning steps]
set -o pipefail
W=${1:-forkjoin-4096x1000-d16}
S=${2:-8}
O=gpurun_out/prof_commit_$W
export TMPDIR=/tmp
mkdir -p $O
WF=/tmp/fate_workload_$W.npz
echo "[profile] generate" && timeout -k 10 300 python3 bench.py --workload $W --workload-file $WF --steps 2 --warmup 1 --no-cpu-baseline --no-medians --no-sweep --no-sim --planning-steps 0 > $O/generate.log 2>&1 || exit $?
echo "[profile] kernel trace" && timeout -k 10 300 rocprofv3 --kernel-trace --stats -d $O/trace -o kt -- python3 bench.py --workload $W --workload-file $WF --steps 2 --warmup 1 --no-cpu-baseline --no-medians --no-sweep --no-sim --planning-steps $S > $O/trace.log 2>&1 || exit $?
python3 -m paper_2605_07238_amd.profile_summary --trace-db $(ls $O/trace/*.db | head -1) > $O/summary.txt || exit $?
grep "planning step" $O/trace.log
cat $O/summary.txt
