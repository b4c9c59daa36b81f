#!/bin/bash
# rocprofv3 runs behind the committed summaries in profiles/ (run from the repository root on
# a GPU host; raw results go to $TASP_PROFILE_OUT, by default ./profile_out).
#   decode_b1:  kernel trace of the default benchmark (8B layer, batch 1), then FETCH_SIZE and
#               WRITE_SIZE passes of its sparse plan
#   decode_b8:  kernel trace and FETCH_SIZE / WRITE_SIZE passes of the batch-8 benchmark
#   decode_b8_busy: VALU and MFMA busy counters of the batch-8 benchmark's sparse plan
#   prefill:    kernel trace and MFMA counter pass of the 512-token prefill benchmark
#   prefill2048: kernel trace of the 2048-token prefill benchmark
#   router:     kernel trace of the router benchmark (one 7 KiB turn, then 512-prompt batches)
#   shared:     kernel trace of the shared-store benchmark (8B layer, batch 1)
#   stack70:    kernel trace of the default benchmark (80-layer 70B stack, seed-1 mask then the
#               dense plan; extras off), then FETCH_SIZE and WRITE_SIZE passes of its sparse plan
#   stack8:     the same three runs for the 32-layer 8B stack (seed-1 mask)
set -o pipefail
export TMPDIR=/tmp
R=$(pwd)
O=${TASP_PROFILE_OUT:-$R/profile_out}
mkdir -p $O
which=${1:-decode_b1}
case $which in
decode_b1)
  echo "[prof] b1 kernel trace" && timeout -k 10 400 rocprofv3 --kernel-trace --stats -d $O/b1_trace -o trace -- python3 -u bench.py --workload llama3_8b_layer --cpu-seconds 3 > $O/b1_trace.json 2> $O/b1_trace.err &&
  echo "[prof] b1 FETCH_SIZE" && timeout -s KILL 300 rocprofv3 --pmc FETCH_SIZE -d $O/b1_fetch -o fetch -- python3 -u bench.py --workload llama3_8b_layer --sparse-only --no-cpu --steps 200 --warmup 20 --blocks 1 --timed-launches 8 > $O/b1_fetch.json 2> $O/b1_fetch.err &&
  echo "[prof] b1 WRITE_SIZE" && timeout -s KILL 300 rocprofv3 --pmc WRITE_SIZE -d $O/b1_write -o write -- python3 -u bench.py --workload llama3_8b_layer --sparse-only --no-cpu --steps 200 --warmup 20 --blocks 1 --timed-launches 8 > $O/b1_write.json 2> $O/b1_write.err
  ;;
decode_b8)
  echo "[prof] b8 kernel trace" && timeout -k 10 400 rocprofv3 --kernel-trace --stats -d $O/b8_trace -o trace -- python3 -u bench.py --workload llama3_8b_batch8 --steps 200 --warmup 20 --cpu-seconds 3 > $O/b8_trace.json 2> $O/b8_trace.err &&
  echo "[prof] b8 FETCH_SIZE" && timeout -s KILL 300 rocprofv3 --pmc FETCH_SIZE -d $O/b8_fetch -o fetch -- python3 -u bench.py --workload llama3_8b_batch8 --sparse-only --no-cpu --steps 100 --warmup 10 --blocks 1 --timed-launches 8 > $O/b8_fetch.json 2> $O/b8_fetch.err &&
  echo "[prof] b8 WRITE_SIZE" && timeout -s KILL 300 rocprofv3 --pmc WRITE_SIZE -d $O/b8_write -o write -- python3 -u bench.py --workload llama3_8b_batch8 --sparse-only --no-cpu --steps 100 --warmup 10 --blocks 1 --timed-launches 8 > $O/b8_write.json 2> $O/b8_write.err
  ;;
decode_b8_busy)
  echo "[prof] b8 VALU / MFMA busy" && timeout -s KILL 300 rocprofv3 --pmc VALUBusy MfmaUtil -d $O/b8_busy -o busy -- python3 -u bench.py --workload llama3_8b_batch8 --sparse-only --no-cpu --steps 100 --warmup 10 --blocks 1 --timed-launches 8 > $O/b8_busy.json 2> $O/b8_busy.err
  ;;
prefill)
  echo "[prof] prefill kernel trace" && timeout -k 10 400 rocprofv3 --kernel-trace --stats -d $O/pf_trace -o trace -- python3 -u bench.py --workload llama3_8b_prefill512 --steps 200 --warmup 20 --cpu-seconds 3 > $O/pf_trace.json 2> $O/pf_trace.err &&
  echo "[prof] prefill MFMA counters" && timeout -s KILL 300 rocprofv3 --pmc MfmaUtil SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_BUSY_CU_CYCLES -d $O/pf_mfma -o mfma -- python3 -u bench.py --workload llama3_8b_prefill512 --no-cpu --steps 40 --warmup 4 > $O/pf_mfma.json 2> $O/pf_mfma.err
  ;;
prefill2048)
  echo "[prof] prefill 2048 kernel trace" && timeout -k 10 400 rocprofv3 --kernel-trace --stats -d $O/pf2k_trace -o trace -- python3 -u bench.py --workload llama3_8b_prefill2048 --steps 50 --warmup 5 --cpu-seconds 3 > $O/pf2k_trace.json 2> $O/pf2k_trace.err
  ;;
router)
  echo "[prof] router kernel trace" && timeout -k 10 400 rocprofv3 --kernel-trace --stats -d $O/rt_trace -o trace -- python3 -u bench.py --workload router_llama3_8b --steps 200 --warmup 20 --cpu-seconds 3 > $O/rt_trace.json 2> $O/rt_trace.err
  ;;
stack70)
  echo "[prof] 70B stack kernel trace" && timeout -k 10 600 rocprofv3 --kernel-trace --stats -d $O/s70_trace -o trace -- python3 -u bench.py --no-extras --steps 40 --warmup 5 --blocks 1 --block-warmup 5 --block-steps 50 --cpu-seconds 3 > $O/s70_trace.json 2> $O/s70_trace.err &&
  echo "[prof] 70B stack FETCH_SIZE" && timeout -s KILL 400 rocprofv3 --pmc FETCH_SIZE -d $O/s70_fetch -o fetch -- python3 -u bench.py --sparse-only --no-cpu --steps 4 --warmup 1 --blocks 0 > $O/s70_fetch.json 2> $O/s70_fetch.err &&
  echo "[prof] 70B stack WRITE_SIZE" && timeout -s KILL 400 rocprofv3 --pmc WRITE_SIZE -d $O/s70_write -o write -- python3 -u bench.py --sparse-only --no-cpu --steps 4 --warmup 1 --blocks 0 > $O/s70_write.json 2> $O/s70_write.err
  ;;
stack8)
  echo "[prof] 8B stack kernel trace" && timeout -k 10 600 rocprofv3 --kernel-trace --stats -d $O/s8_trace -o trace -- python3 -u bench.py --workload llama3_8b_stack --steps 40 --warmup 5 --blocks 1 --block-warmup 5 --block-steps 50 --cpu-seconds 3 > $O/s8_trace.json 2> $O/s8_trace.err &&
  echo "[prof] 8B stack FETCH_SIZE" && timeout -s KILL 400 rocprofv3 --pmc FETCH_SIZE -d $O/s8_fetch -o fetch -- python3 -u bench.py --workload llama3_8b_stack --sparse-only --no-cpu --steps 4 --warmup 1 --blocks 0 > $O/s8_fetch.json 2> $O/s8_fetch.err &&
  echo "[prof] 8B stack WRITE_SIZE" && timeout -s KILL 400 rocprofv3 --pmc WRITE_SIZE -d $O/s8_write -o write -- python3 -u bench.py --workload llama3_8b_stack --sparse-only --no-cpu --steps 4 --warmup 1 --blocks 0 > $O/s8_write.json 2> $O/s8_write.err
  ;;
shared)
  echo "[prof] shared kernel trace" && timeout -k 10 400 rocprofv3 --kernel-trace --stats -d $O/sh_trace -o trace -- python3 -u bench.py --workload llama3_8b_layer_shared --steps 200 --warmup 20 --cpu-seconds 3 > $O/sh_trace.json 2> $O/sh_trace.err
  ;;
esac
