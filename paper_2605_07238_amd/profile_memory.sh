#!/bin/bash
# Memory-pipeline counters of the benchmark's score kernel: two --pmc passes
# (wave waits, vector-memory instructions and address-unit activity; then L1
# and L2 request, latency and hit counts) over the same rotated-copy run as
# profile_run.sh.  Writes raw output under gpurun_out/mem_<workload>/ and
# prints the summary.
#   usage: paper_2605_07238_amd/profile_memory.sh <workload> [steps]
set -o pipefail
W=${1:-forkjoin-4096x1000-d16}
S=${2:-10}
O=gpurun_out/mem_$W
export TMPDIR=/tmp
mkdir -p $O
WF=/tmp/fate_workload_$W.npz
echo "[profile] generate" && timeout -k 10 300 python3 bench.py --workload $W --workload-file $WF --steps 2 --warmup 1 --no-cpu-baseline --no-sweep --no-sim --planning-steps 0 > $O/generate.log 2>&1 || exit $?
B="python3 bench.py --workload $W --workload-file $WF --steps $S --warmup 2 --no-cpu-baseline --no-medians --no-warm --no-sweep --no-sim --planning-steps 0"
echo "[profile] SQ/TA/TD pass" && timeout -s KILL 180 rocprofv3 --pmc SQ_INSTS_VMEM_RD SQ_INSTS_VMEM_WR SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_WAVE_CYCLES SQ_BUSY_CU_CYCLES GRBM_GUI_ACTIVE TA_BUSY_avr TD_BUSY_sum -d $O/sq -o pmc --output-format csv -- $B > $O/sq.log 2>&1 || exit $?
echo "[profile] TCP/TCC pass" && timeout -s KILL 180 rocprofv3 --pmc TCP_TCC_READ_REQ_sum TCP_TCC_READ_REQ_LATENCY_sum TCP_TOTAL_CACHE_ACCESSES_sum TCP_PENDING_STALL_CYCLES_sum TCC_HIT_sum TCC_MISS_sum GRBM_GUI_ACTIVE -d $O/tcp -o pmc --output-format csv -- $B > $O/tcp.log 2>&1 || exit $?
python3 -m paper_2605_07238_amd.profile_summary \
  --pmc $O/sq/pmc_counter_collection.csv $O/tcp/pmc_counter_collection.csv \
  --kernel-source paper_2605_07238_amd/csrc/fate_kernels.hip paper_2605_07238_amd/csrc/fate_internal.h > $O/summary.txt || exit $?
cat $O/summary.txt
