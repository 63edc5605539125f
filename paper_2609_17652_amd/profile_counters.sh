#!/bin/bash
# Hardware-counter passes behind profiles/scan_topk_layer1m_b48_{sq,traffic}.json:
# three SQ passes (8 SQ counters at most each) and FETCH_SIZE / WRITE_SIZE
# (one pass each), every pass its own short bench run, then the summaries.
# Usage (MI355X, from the repository root): bash paper_2609_17652_amd/profile_counters.sh OUTDIR
set -o pipefail
R=$(pwd)
OUT=${1:-$R/gpurun_out/counters}
mkdir -p "$OUT"
OUT=$(cd "$OUT" && pwd)  # absolute: the passes run from /tmp
BENCH="python3 $R/bench.py --steps 3 --warmup 1 --scan-reps 2 --copies 2 --no-cpu-baseline --traffic-calib 256"
PASSES=(
  "SQ_WAVES,SQ_WAVE_CYCLES,SQ_BUSY_CYCLES,SQ_WAIT_ANY,SQ_INSTS_VALU,SQ_INSTS_SALU,SQ_INSTS_LDS,SQ_INSTS_VMEM_RD"
  "SQ_ACTIVE_INST_VALU,SQ_ACTIVE_INST_LDS,SQ_ACTIVE_INST_SCA,SQ_INSTS_MFMA,SQ_WAIT_INST_ANY,SQ_WAIT_INST_LDS,SQ_INSTS_BRANCH,SQ_ACTIVE_INST_MISC"
  "SQ_LDS_BANK_CONFLICT,SQ_LDS_IDX_ACTIVE,SQ_LDS_ADDR_CONFLICT,SQ_VALU_MFMA_BUSY_CYCLES,SQ_INSTS_SMEM,SQ_IFETCH,SQ_INST_CYCLES_SALU,SQ_INSTS_VALU_MFMA_I8"
  "FETCH_SIZE"
  "WRITE_SIZE"
)
cd /tmp && export TMPDIR=/tmp
i=0
for c in "${PASSES[@]}"; do
  echo "[counters] pass $i: $c"; date
  timeout -s KILL 120 rocprofv3 --pmc ${c//,/ } --output-format csv -d "$OUT/p$i" -o p -- $BENCH > "$OUT/p$i.log" 2>&1
  rc=$?; tail -1 "$OUT/p$i.log"; [ $rc -eq 0 ] || exit $rc
  i=$((i + 1))
done
cd "$R"
python3 bench.py --sq-summary "$OUT/p0/p_counter_collection.csv" "$OUT/p1/p_counter_collection.csv" \
  "$OUT/p2/p_counter_collection.csv" > "$OUT/sq.json" && \
python3 bench.py --traffic-calib 256 --traffic-summary "$OUT/p3/p_counter_collection.csv" \
  "$OUT/p4/p_counter_collection.csv" > "$OUT/traffic.json"
