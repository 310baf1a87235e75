#!/bin/bash
# Profiles bench.py's tuned GEMM with rocprofv3 into OUT (default ./profile_out):
#   1. the whole bench step under --kernel-trace --stats (the search and the re-timed best);
#   2. FETCH_SIZE, then WRITE_SIZE, on the best configuration replayed 20 times;
#   3. the same two counters on a plain 1 GiB device copy (their byte scale);
#   4. MFMA-busy, LDS and wait counters on the replayed best configuration.
# Then: python3 paper_1909_10616_amd/profsum.py report OUT > profiles/<name>.md
# Usage: profile_bench.sh [OUT] [extra bench.py arguments, e.g. --workload NAME]
set -u
ROOT=$(cd "$(dirname "$0")/.." && pwd)
OUT=$(realpath -m "${1:-$ROOT/profile_out}")
shift || true
export TMPDIR=/tmp
mkdir -p "$OUT"
cd /tmp
echo "profile: bench under kernel trace -> $OUT/trace"
timeout -k 10 400 rocprofv3 --kernel-trace --stats --output-format csv -d "$OUT/trace" -o bench -- \
  python3 "$ROOT/bench.py" --no-cpu-baseline "$@" > "$OUT/bench_traced.json" 2> "$OUT/bench_traced.err" || exit $?
CFG=$(python3 "$ROOT/paper_1909_10616_amd/profsum.py" bestcfg "$OUT/bench_traced.json") || exit $?
echo "profile: best configuration $CFG"
timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE --output-format csv -d "$OUT/fetch" -o k -- \
  python3 "$ROOT/bench.py" "$@" --replay "$CFG" --repeat 20 > "$OUT/replay_fetch.json" || exit $?
timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE --output-format csv -d "$OUT/write" -o k -- \
  python3 "$ROOT/bench.py" "$@" --replay "$CFG" --repeat 20 > "$OUT/replay_write.json" || exit $?
echo "profile: copy calibration"
timeout -s KILL 120 rocprofv3 --pmc FETCH_SIZE --output-format csv -d "$OUT/cfetch" -o c -- \
  python3 "$ROOT/bench.py" --calibrate-copy 1024 --repeat 5 > "$OUT/copy_fetch.json" || exit $?
timeout -s KILL 120 rocprofv3 --pmc WRITE_SIZE --output-format csv -d "$OUT/cwrite" -o c -- \
  python3 "$ROOT/bench.py" --calibrate-copy 1024 --repeat 5 > "$OUT/copy_write.json" || exit $?
echo "profile: utilisation counters"
timeout -s KILL 120 rocprofv3 --pmc SQ_VALU_MFMA_BUSY_CYCLES GRBM_GUI_ACTIVE SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE \
  SQ_WAVE_CYCLES SQ_WAIT_ANY --output-format csv -d "$OUT/util" -o u -- \
  python3 "$ROOT/bench.py" "$@" --replay "$CFG" --repeat 20 > "$OUT/replay_util.json" || exit $?
echo "profile: done"
