#!/bin/bash
# rocprofv3 runs behind the committed profile summaries (run from the
# repository root on an MI355X host): kernel trace with statistics of the
# benchmark's step, HBM traffic counters (one counter per pass) with the
# calibration copy, and compute-side counters; an entry overlap:W profiles the
# overlap round's multi-branch attention on workload W instead (trace and
# traffic).  Usage:
#   bash paper_2609_34388_amd/profile_runs.sh <out-dir> <workload | overlap:workload> [...]
set -u
OUT=$(realpath "$1"); shift
REPO=$(pwd)
BENCH="$REPO/bench.py --no-block-sizing --no-cpu-baseline --no-all-configs"
cd /tmp && export TMPDIR=/tmp
mkdir -p "$OUT"
for c in FETCH_SIZE WRITE_SIZE; do
  echo "[profile] copy calibration $c"
  timeout -s KILL 120 rocprofv3 --pmc $c --output-format csv -d "$OUT/copy_$c" -o copy -- python3 $REPO/bench.py --copy-calibration-mb 256 > "$OUT/copy_$c.log" 2>&1 || exit 1
done
for entry in "$@"; do
  case $entry in
    overlap:*) wl=${entry#overlap:}; tag=overlap_$wl; ARGS="$BENCH --no-quadratic --workload $wl" ;;
    *) wl=$entry; tag=$wl; ARGS="$BENCH --no-overlap --workload $wl" ;;
  esac
  echo "[profile] kernel trace $tag"
  timeout -k 10 300 rocprofv3 --kernel-trace --stats --output-format csv -d "$OUT/trace_$tag" -o $tag -- python3 $ARGS --steps 20 --warmup 5 > "$OUT/trace_$tag.log" 2>&1 || exit 1
  for c in FETCH_SIZE WRITE_SIZE; do
    echo "[profile] $c $tag"
    timeout -s KILL 240 rocprofv3 --pmc $c --output-format csv -d "$OUT/pmc_${c}_$tag" -o $tag -- python3 $ARGS --steps 3 --warmup 1 > "$OUT/pmc_${c}_$tag.log" 2>&1 || exit 1
  done
  case $entry in overlap:*) continue ;; esac
  echo "[profile] SQ counters $tag"
  timeout -s KILL 240 rocprofv3 --pmc SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_VALU_MFMA_BUSY_CYCLES SQ_BUSY_CU_CYCLES SQ_INSTS_VALU SQ_INSTS_LDS SQ_LDS_BANK_CONFLICT SQ_WAVE_CYCLES GRBM_GUI_ACTIVE --output-format csv -d "$OUT/sq_$tag" -o $tag -- python3 $ARGS --steps 3 --warmup 1 > "$OUT/sq_$tag.log" 2>&1 || exit 1
done
echo "[profile] done"
