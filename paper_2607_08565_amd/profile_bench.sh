#!/bin/bash
# The profiles under profiles/: a rocprofv3 kernel trace of the benchmark command
# (bench.py --gpus 1 --steps 20 --warmup 5), then one FETCH_SIZE and one WRITE_SIZE counter
# run of the same command with --calibrate-copy (a 1 GiB device copy after the timed steps
# fixes the counters' scale), summarised by bench.py itself.  Run from the repository root
# on an MI355X; raw output goes to $PROFILE_OUT (default: profile_out/ in the repository).
# Usage: profile_bench.sh [trace|counters|all|sq]  (sq: one run with the SQ instruction
# counters, summarised per kernel).
set -o pipefail
R=$(pwd)
O=${PROFILE_OUT:-$R/profile_out}
case $O in /*) ;; *) O=$R/$O ;; esac
mkdir -p $O
CMD="$R/bench.py --gpus 1 --steps 20 --warmup 5"
STAGE=${1:-all}
cd /tmp && export TMPDIR=/tmp
if [ $STAGE = trace ] || [ $STAGE = all ]; then
echo "== kernel trace: python3 bench.py --gpus 1 --steps 20 --warmup 5"
timeout -k 10 900 rocprofv3 --kernel-trace --stats --output-format csv -d $O/trace -o run -- python3 $CMD \
  > $O/trace_bench.log 2>&1 || { tail -5 $O/trace_bench.log; exit 2; }
T=$(find $O/trace -name "*kernel_trace.csv" | head -1)
S=$(find $O/trace -name "*kernel_stats.csv" | head -1)
cd $R && python3 bench.py --summarize-trace $T --steps 20 > $O/trace_summary.md || exit 5
cp $S $O/kernel_stats.csv
grep '^{"metric"' $O/trace_bench.log | tail -1 > $O/bench_line.json
cd /tmp
fi
if [ $STAGE = counters ] || [ $STAGE = all ]; then
echo "== FETCH_SIZE"
timeout -s KILL 900 rocprofv3 --pmc FETCH_SIZE --output-format csv -d $O/fetch -o run -- python3 $CMD --calibrate-copy \
  > $O/fetch_bench.log 2>&1 || { tail -5 $O/fetch_bench.log; exit 3; }
echo "== WRITE_SIZE"
timeout -s KILL 900 rocprofv3 --pmc WRITE_SIZE --output-format csv -d $O/write -o run -- python3 $CMD --calibrate-copy \
  > $O/write_bench.log 2>&1 || { tail -5 $O/write_bench.log; exit 4; }
cd $R
F=$(find $O/fetch -name "*counter_collection.csv" | head -1)
W=$(find $O/write -name "*counter_collection.csv" | head -1)
python3 bench.py --summarize-pmc $F $W $O/fetch_bench.log --steps 20 --traffic $O/traffic.json > $O/traffic_summary.md || exit 6
fi
if [ $STAGE = sq ]; then
echo "== SQ instruction counters"
timeout -s KILL 900 rocprofv3 --pmc SQ_WAVES SQ_INSTS_VALU SQ_INSTS_SALU SQ_INSTS_LDS SQ_INSTS_VMEM_RD SQ_INSTS_VMEM_WR \
  SQ_WAVE_CYCLES --output-format csv -d $O/sq -o run -- python3 $CMD > $O/sq_bench.log 2>&1 || { tail -5 $O/sq_bench.log; exit 7; }
cd $R
Q=$(find $O/sq -name "*counter_collection.csv" | head -1)
python3 bench.py --summarize-sq $Q $O/sq_bench.log --steps 20 > $O/sq_summary.md || exit 8
fi
echo "done"
