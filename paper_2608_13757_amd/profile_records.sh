#!/bin/bash
# Writes profiles/<kernel>_traffic.json and profiles/<kernel>_kernel_trace.md
# from the rocprofv3 output of these runs under one output root R (repository
# root, TMPDIR=/tmp):
#   rocprofv3 --kernel-trace --stats --output-format csv -d $R/pt_$wl -o t -- python -u bench.py --workload $wl --steps 50 --warmup 50 --modes barrier_free,barrier --no-cpu-baseline
#   rocprofv3 --pmc FETCH_SIZE --output-format csv -d $R/pf_$wl -o f -- python -u bench.py --workload $wl --steps 2 --warmup 1 --modes barrier_free --no-cpu-baseline --copy-calibration-mib 1024
#   rocprofv3 --pmc WRITE_SIZE --output-format csv -d $R/pw_$wl -o w -- python -u bench.py --workload $wl --steps 2 --warmup 1 --modes barrier_free --no-cpu-baseline --copy-calibration-mib 1024
#   rocprofv3 --pmc $SQ1 --output-format csv -d $R/ps1_$wl -o s -- python -u bench.py --workload $wl --steps 2 --warmup 1 --modes barrier_free,barrier --no-cpu-baseline
#   rocprofv3 --pmc $SQ2 --output-format csv -d $R/ps2_$wl -o s -- python -u bench.py --workload $wl --steps 2 --warmup 1 --modes barrier_free,barrier --no-cpu-baseline
# (SQ1, SQ2 below; the SQ records are written when those runs exist)
# for wl in stream gemm attn moe rmsnorm adamw, and the trace run alone for
# chain (one workgroup, latency-bound: no traffic or SQ record).  The
# algorithmic bytes per step come from bench.py --algorithmic-bytes (the same
# count the benchmark divides by).
set -e
R=${1:?usage: profile_records.sh <rocprofv3 output root>}
SQ1="SQ_WAVES SQ_WAVE_CYCLES SQ_BUSY_CYCLES SQ_WAIT_ANY SQ_WAIT_INST_ANY SQ_ACTIVE_INST_ANY SQ_INSTS_SALU SQ_INSTS_LDS"
SQ2="SQ_INSTS_VALU SQ_INSTS_MFMA SQ_VALU_MFMA_BUSY_CYCLES SQ_INSTS_VALU_MFMA_MOPS_BF16 SQ_INSTS_BRANCH SQ_INSTS_SMEM SQ_LDS_BANK_CONFLICT SQ_LDS_IDX_ACTIVE GRBM_GUI_ACTIVE"
for wl in ${WLS:-stream gemm attn moe rmsnorm adamw}; do
  case $wl in
    stream) k=stream3; wk="sync-bound stream, 1024 workgroups, seed 0, 5568928 innermost iterations, one in-place ring";;
    gemm) k=gemm; wk="GEMM + bias + GELU 4096^3 bf16, seed 0";;
    attn) k=attn; wk="varlen attention forward, 32 sequences U[128,4096] (81588 tokens), 16 heads x 128, seed 0";;
    adamw) k=adamw; wk="AdamW step, 2^20 fp32 parameters, 512 workgroups of 2 chunks of 1024, 2 vector waves, 2-slot ring, seed 0";;
    rmsnorm) k=rms; wk="RMSNorm + FP8 E4M3 quantization, 32768 x 8192 bf16, 768 workgroups, 4 vector waves, rings 2 + 2, seed 0";;
    moe) k=moe; wk="MoE grouped GEMM, 32768 tokens, 64 Zipf(1.1) experts, hidden 4096, ffn 1408, M-tiles of 256 tokens, seed 0 (both launches)";;
    chain) k=chain; wk="two-engine chain, 1 workgroup, loop A of 16 iterations, inner trips U[1,8], 4-slot ring, seeds 0, 1, 2, on its own kernel and on the interpreter";;
  esac
  if [ $wl != chain ]; then
  ab=$(python bench.py --workload $wl --algorithmic-bytes)
  python -m paper_2608_13757_amd.profiles traffic --kernel $k --fetch-dir $R/pf_$wl --write-dir $R/pw_$wl --copy-mib 1024 \
    --algorithmic-bytes $ab --workload "$wk" \
    --command "rocprofv3 --pmc FETCH_SIZE --output-format csv -d $R/pf_$wl -o f -- python -u bench.py --workload $wl --steps 2 --warmup 1 --modes barrier_free --no-cpu-baseline --copy-calibration-mib 1024" \
    --command "rocprofv3 --pmc WRITE_SIZE --output-format csv -d $R/pw_$wl -o w -- python -u bench.py --workload $wl --steps 2 --warmup 1 --modes barrier_free --no-cpu-baseline --copy-calibration-mib 1024" \
    --command "WLS=$wl bash paper_2608_13757_amd/profile_records.sh $R"
  if [ -d $R/ps1_$wl ] && [ -d $R/ps2_$wl ]; then
    python -m paper_2608_13757_amd.profiles sq --kernel $k --dir $R/ps1_$wl --dir $R/ps2_$wl --workload "$wk" \
      --command "rocprofv3 --pmc $SQ1 --output-format csv -d $R/ps1_$wl -o s -- python -u bench.py --workload $wl --steps 2 --warmup 1 --modes barrier_free,barrier --no-cpu-baseline" \
      --command "rocprofv3 --pmc $SQ2 --output-format csv -d $R/ps2_$wl -o s -- python -u bench.py --workload $wl --steps 2 --warmup 1 --modes barrier_free,barrier --no-cpu-baseline" \
      --command "WLS=$wl bash paper_2608_13757_amd/profile_records.sh $R"
  fi
  fi
  python -m paper_2608_13757_amd.profiles trace --kernel $k --stats-dir $R/pt_$wl --workload "$wk" \
    --command "rocprofv3 --kernel-trace --stats --output-format csv -d $R/pt_$wl -o t -- python -u bench.py --workload $wl --steps 50 --warmup 50 --modes barrier_free,barrier --no-cpu-baseline" \
    --command "WLS=$wl bash paper_2608_13757_amd/profile_records.sh $R"
done
