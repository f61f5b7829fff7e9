#!/bin/bash
# Profile the benchmark's score kernel with rocprofv3: one kernel-trace run
# and two counter passes (FETCH_SIZE, WRITE_SIZE), each ending with a plain
# 512 MiB device copy for counter calibration.  Writes raw output under
# gpurun_out/prof_<workload>/ and prints the summaries.
#   usage: paper_2605_07238_amd/profile_run.sh <workload> [steps]
set -o pipefail
W=${1:-forkjoin-4096x1000-d16}
S=${2:-10}
O=gpurun_out/prof_$W
export TMPDIR=/tmp
mkdir -p $O
WF=/tmp/fate_workload_$W.npz
# generate once, unprofiled (the generator forks worker processes); the
# profiled runs load the saved batch
echo "[profile] generate" && timeout -k 10 300 python3 bench.py --workload $W --workload-file $WF --steps 2 --warmup 1 --no-cpu-baseline --no-sweep --no-sim --planning-steps 0 > $O/generate.log 2>&1 || exit $?
B="python3 bench.py --workload $W --workload-file $WF --steps $S --warmup 2 --no-cpu-baseline --no-medians --no-warm --no-sweep --no-sim --planning-steps 0 --copy-calibration"
echo "[profile] kernel trace" && timeout -k 10 300 rocprofv3 --kernel-trace --stats -d $O/trace -o kt -- $B > $O/trace.log 2>&1 || exit $?
echo "[profile] FETCH_SIZE" && timeout -s KILL 180 rocprofv3 --pmc FETCH_SIZE -d $O/fetch -o pmc --output-format csv -- $B > $O/fetch.log 2>&1 || exit $?
echo "[profile] WRITE_SIZE" && timeout -s KILL 180 rocprofv3 --pmc WRITE_SIZE -d $O/write -o pmc --output-format csv -- $B > $O/write.log 2>&1 || exit $?
echo "[profile] SQ counters" && timeout -s KILL 180 rocprofv3 --pmc SQ_WAVES SQ_BUSY_CYCLES SQ_WAVE_CYCLES SQ_INSTS_VALU SQ_ACTIVE_INST_VALU SQ_INSTS_LDS SQ_INSTS_SALU GRBM_GUI_ACTIVE -d $O/sq -o pmc --output-format csv -- $B > $O/sq.log 2>&1 || exit $?
python3 -m paper_2605_07238_amd.profile_summary --trace-db $(ls $O/trace/*.db | head -1) \
  --pmc $O/fetch/pmc_counter_collection.csv $O/write/pmc_counter_collection.csv $O/sq/pmc_counter_collection.csv \
  --kernel-source paper_2605_07238_amd/csrc/fate_kernels.hip paper_2605_07238_amd/csrc/fate_internal.h > $O/summary.txt || exit $?
grep "timed" $O/trace.log | head -2
cat $O/summary.txt
