"""Benchmark of the barrier-free synchronization hot path on one MI355X.

Workload (the sync-bound microbenchmark): three engines -- HBM->LDS load,
vector add, LDS->HBM store -- over a 3-level dynamically bounded nest with
outer trip 256, middle trips uniform in [1, 16] and inner trips uniform in
[1, 4] (per workgroup seed), 64-element fp32 tiles, 1024 independent
workgroups.  One step = one launch over all workgroups.  The same program
runs in barrier mode (drain + barrier + reset at every loop entry and
iteration end) as the in-run comparison.

Prints one JSON line: value = sync-bound ops/s of the barrier-free mode
(3 engine operations per innermost iteration), with the barrier-mode latency
and speedup, the HBM roofline of the stream kernel and the CPU oracle timed
on the host.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "latency vs all-barrier baseline (us); sync-bound ops/s; % of HBM/MFMA peak"
HBM_PEAK_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--n-wg", type=int, default=1024)
    ap.add_argument("--outer", type=int, default=256)
    ap.add_argument("--n-gen", type=int, default=32)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-measured-peak", action="store_true",
                    help="skip the copy / library-matmul measurement of achievable peaks")
    ap.add_argument("--modes", default="barrier_free,barrier")
    ap.add_argument("--moe-ring", default="linear", choices=["linear", "acq"],
                    help="MoE: protect the load ring across M-tiles with the linearized MMA->LOAD dependency "
                         "(an extension of the paper's relation) or with the paper's acquire instruction that "
                         "drains the ring at every M-tile (MMA->ACQL, k = 1)")
    ap.add_argument("--k-unroll", type=int, default=0, choices=[0, 1, 2, 4, 8],
                    help="GEMM: K steps per copy of the loop bodies (static-trip unrolling)")
    ap.add_argument("--alloc", default="per_loop", choices=["per_loop", "per_instr"],
                    help="counter allocation of the barrier-free plans (Eq. 5 per loop and engine, "
                         "or Eq. 3 one counter per producer instruction)")
    ap.add_argument("--workload", default="stream", choices=["stream", "gemm", "attn", "moe", "rmsnorm", "adamw", "ring"],
                    help="stream: the sync-bound microbenchmark (headline); gemm: 4096^3 bf16 GEMM + bias + GELU; "
                         "attn: varlen attention forward; moe: MoE grouped GEMM; rmsnorm: RMSNorm + FP8 "
                         "quantization of 32768 x 8192 bf16; adamw: AdamW step over fp32 parameters; ring: "
                         "a ring indexed across trips on the interpreter, drained by an ACQ at every trip start "
                         "(the paper's form) vs one linearized-offset dependency (an extension)")
    ap.add_argument("--adam-params", type=int, default=1 << 20, help="adamw: parameters (the paper's 2^20 by default)")
    ap.add_argument("--adam-wg", type=int, default=0, help="adamw: workgroups (0: one per 2 chunks, at most 1024)")
    ap.add_argument("--adam-chunk", type=int, default=1024, help="adamw: parameters per chunk (256, 512, 1024)")
    ap.add_argument("--adam-waves", type=int, default=2, help="adamw: vector-engine waves")
    ap.add_argument("--adam-ring", type=int, default=2, help="adamw: ring slots")
    ap.add_argument("--rms-wg", type=int, default=768, help="rmsnorm: workgroups (3 per CU)")
    ap.add_argument("--rms-waves", type=int, default=4, help="rmsnorm: vector-engine waves sharing each row")
    ap.add_argument("--rms-ring", default="2,2", help="rmsnorm: x-ring and q-ring slots")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the timed region, run one plain device copy of this many MiB "
                         "(reference dispatch for HBM traffic counters)")
    return ap.parse_args()


def alloc_of(a, mode):
    """Counter allocation of a plan: the requested one for barrier-free plans
    (barrier mode keeps its one counter per engine)."""
    from paper_2608_13757_amd import ALLOC_PER_INSTR, ALLOC_PER_LOOP, MODE_BARRIER_FREE
    if mode != MODE_BARRIER_FREE:
        return ALLOC_PER_LOOP
    return ALLOC_PER_INSTR if a.alloc == "per_instr" else ALLOC_PER_LOOP


def time_mode(plan, bufs, trips, toff, n_wg, steps, warmup, **run_kw):
    import torch
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        plan.run(bufs, trips, toff, n_wg, stream=stream, **run_kw)
    plan.status(stream)
    starts = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(steps):
        starts[i].record(stream)
        plan.run(bufs, trips, toff, n_wg, stream=stream, **run_kw)
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    plan.status(stream)
    per = [s.elapsed_time(e) for s, e in zip(starts, ends)]   # ms, per launch
    return {"ms_mean": sum(per) / len(per), "ms_min": min(per), "ms_median": sorted(per)[len(per) // 2],
            "wall_ms_per_step": 1e3 * wall / steps}


def measured_peak(bound):
    """Achievable rates measured on this GPU next to the vendor peaks: a
    device-to-device copy of 1 GiB (bytes read + written per second) for
    HBM-bound kernels, the vendor library's bf16 matmul at 4096^3 and 8192^3
    for MFMA-bound ones."""
    import torch

    def timed(fn, reps):
        for _ in range(2):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3
    if bound == "hbm":
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        t = timed(lambda: dst.copy_(src), 5)
        del src, dst
        return {"copy_1GiB_gbs": 2.0 * (1 << 30) / t / 1e9}
    res = {}
    for n in (4096, 8192):
        x = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
        w = torch.randn(n, n, device="cuda", dtype=torch.bfloat16)
        t = timed(lambda: torch.matmul(x, w), 10)
        res[f"library_bf16_matmul_{n}_tflops"] = 2.0 * n ** 3 / t / 1e12
        del x, w
    return res


def emit(out, a, kernel):
    """Attach the recorded HBM traffic of the kernel (when its profile matches
    the current sources) and the achievable peaks measured on this GPU, run
    the copy that calibrates traffic counters if asked, and print the JSON
    line."""
    import torch
    from paper_2608_13757_amd.profiles import recorded_traffic
    tr = recorded_traffic(kernel)
    if tr is not None:
        out["roofline"]["traffic"] = tr
    if not a.no_measured_peak:
        mp = measured_peak(out["roofline"]["bound"])
        best = max(mp.values())
        mp["frac_of_measured"] = out["roofline"]["achieved"] / best
        out["measured_peak"] = mp
    if a.copy_calibration_mib:
        src = torch.empty(a.copy_calibration_mib << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
    print(json.dumps(out), flush=True)


def cpu_baseline(w, budget_s=20.0):
    """The CPU oracle's sequential program-order execution of the same
    workload (fp64 values), single-threaded, on as many workgroups as fit in
    the time budget."""
    import numpy as np
    from oracle import core
    trips, off = w.trips.flat()
    n_wg = w.trips.n_wg
    done, iters, t_used = 0, 0, 0.0
    chunk = 16
    while done < n_wg and t_used < budget_s:
        hi = min(n_wg, done + chunk)
        sub_off = off[done:hi]
        base = w.base[done:hi] - w.base[done]
        n_t = int(w.counts[done:hi].sum())
        x = w.x[w.base[done]:w.base[done] + n_t]
        t0 = time.perf_counter()
        core.values(w.prog, trips, sub_off, base, x, n_t * 64)
        t_used += time.perf_counter() - t0
        iters += n_t
        done = hi
    return {"value": 3.0 * iters / t_used, "unit": "ops/s", "cores": 1, "kind": "oracle",
            "sample": f"{done} of {n_wg} workgroups ({iters} innermost iterations, {t_used:.1f} s)"}


MFMA_BF16_PEAK_TFLOPS = 2500.0


def bench_gemm(a):
    """4096^3 bf16 GEMM + bias + GELU, one 256 x 256 tile per workgroup,
    load / MFMA / epilogue engines; both synchronization modes."""
    import numpy as np
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import GEMM_BK, GEMM_RING, gemm_program, gemm_trips
    from workloads.tensors import gemm_inputs

    m = n = k = 4096
    gi = gemm_inputs(seed=a.seed, m=m, n=n, k=k)
    dev = lambda bits: torch.from_numpy(bits.view(np.int16)).cuda()
    A, Bt = dev(gi.a), dev(gi.bt)
    bias = torch.from_numpy(gi.bias).cuda()
    C = torch.empty(m * n, dtype=torch.int16, device="cuda")
    tt = gemm_trips(m, n, k)
    t_np, o_np = tt.flat()
    trips, toff = torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda()
    res = {}
    for name in a.modes.split(","):
        mode = MODE_BARRIER_FREE if name == "barrier_free" else MODE_BARRIER
        plan = Plan(gemm_program(m, n, k), mode, alloc_of(a, mode))
        res[name] = time_mode(plan, [A, Bt, bias, C], trips, toff, tt.n_wg, a.steps, a.warmup,
                              k_unroll=a.k_unroll)
    flop = 2.0 * m * n * k
    bf = res.get("barrier_free", next(iter(res.values())))
    ms = bf["ms_mean"]
    tflops = flop / (ms * 1e-3) / 1e12
    # context: the vendor library's bf16 matmul at the same shape (no bias / GELU)
    x = torch.from_numpy(bf16_bits_as_f32(gi.a)).cuda().to(torch.bfloat16).reshape(m, k)
    w = torch.from_numpy(bf16_bits_as_f32(gi.bt)).cuda().to(torch.bfloat16).reshape(n, k)
    wt = w.t().contiguous()
    for _ in range(3):
        torch.matmul(x, wt)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        torch.matmul(x, wt)
    e1.record()
    torch.cuda.synchronize()
    lib_ms = e0.elapsed_time(e1) / 10
    out = {
        "metric": METRIC, "value": tflops, "unit": "TFLOP/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "GEMM + bias + GELU, A, B bf16 4096 x 4096 ~ N(0,1)/64, 256 x 256 tiles, "
                               f"K steps of {GEMM_BK} through a {GEMM_RING}-slot LDS ring", "m": m, "n": n, "k": k,
                   "k_unroll": a.k_unroll or 1, "parallelism": "single GPU"},
        "latency_us": {kk: v["ms_mean"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / MFMA_BF16_PEAK_TFLOPS, "traffic": None},
        "library_matmul_tflops": flop / (lib_ms * 1e-3) / 1e12,
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    emit(out, a, "gemm")


def bench_attn(a):
    """Variable-length attention forward: 32 sequences of U[128, 4096] tokens,
    16 heads of 128; 256 workgroups (one per compute unit) each run a list of
    (sequence, head, 128-query tile) tiles; both synchronization modes."""
    import numpy as np
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import attn_program, attn_worklist
    from workloads.tensors import attn_inputs

    heads = 16
    ai = attn_inputs(seed=a.seed, heads=heads)
    wl = attn_worklist(ai.lengths, heads)
    dev = lambda bits: torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()
    q, k, v = dev(ai.q), dev(ai.k), dev(ai.v)
    o = torch.empty(ai.q.shape, dtype=torch.int16, device="cuda")
    work = torch.from_numpy(wl.work.reshape(-1)).cuda()
    t_np, o_np = wl.trips.flat()
    trips, toff = torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda()
    res = {}
    for name in a.modes.split(","):
        mode = MODE_BARRIER_FREE if name == "barrier_free" else MODE_BARRIER
        plan = Plan(attn_program(heads), mode, alloc_of(a, mode))
        res[name] = time_mode(plan, [work, q, k, v, o], trips, toff, wl.trips.n_wg, a.steps, a.warmup)
    lens = ai.lengths.astype(np.float64)
    flop = 4.0 * 128 * heads * float(np.sum(lens * lens))
    bf = res.get("barrier_free", next(iter(res.values())))
    ms = bf["ms_mean"]
    tflops = flop / (ms * 1e-3) / 1e12
    out = {
        "metric": METRIC, "value": tflops, "unit": "TFLOP/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "varlen attention forward, 32 sequences of U[128,4096] tokens (seed "
                               f"{a.seed}: {int(lens.sum())} tokens), 16 heads x 128, bf16 N(0,1), "
                               "KV blocks of 64, 128-query tiles", "batch": 32, "heads": heads,
                   "head_dim": 128, "tokens": int(lens.sum()), "n_wg": wl.trips.n_wg,
                   "parallelism": "single GPU"},
        "latency_us": {kk: v["ms_mean"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / MFMA_BF16_PEAK_TFLOPS, "traffic": None},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    emit(out, a, "attn")


def bench_moe(a):
    """MoE grouped GEMM: 32768 tokens routed top-1 to 64 experts with Zipf(1.1)
    counts, hidden 4096, ffn 1408, SiLU-gated; one step = the gate/up launch
    plus the down launch; both synchronization modes."""
    import numpy as np
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import moe_program, moe_worklist
    from workloads.tensors import moe_inputs, moe_weights_all

    moe = moe_inputs(seed=a.seed)
    H, F = moe.hidden, moe.ffn
    dev = lambda bits: torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()
    wg, wu, wd = (dev(w) for w in moe_weights_all(moe))
    x = dev(moe.x)
    perm = torch.from_numpy(moe.perm.astype(np.int32)).cuda()
    eoff = torch.from_numpy(moe.expert_off.astype(np.int32)).cuda()
    T = len(moe.assign)
    h = torch.empty((T, F), dtype=torch.int16, device="cuda")
    y = torch.empty((T, H), dtype=torch.int16, device="cuda")
    launches = {}
    for ph in (1, 2):
        wl = moe_worklist(moe.counts, ph, H, F)
        t_np, o_np = wl.trips.flat()
        work = torch.from_numpy(wl.work.reshape(-1)).cuda()
        bufs = [work, perm, eoff, x, wg, wu, h] if ph == 1 else [work, perm, eoff, h, wd, y]
        launches[ph] = (bufs, torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda(), wl.trips.n_wg)
    stream = torch.cuda.current_stream()
    res = {}
    for name in a.modes.split(","):
        mode = MODE_BARRIER_FREE if name == "barrier_free" else MODE_BARRIER
        plans = {ph: Plan(moe_program(ph, H, F, linear=a.moe_ring == "linear"), mode, alloc_of(a, mode))
                 for ph in (1, 2)}

        def step():
            for ph in (1, 2):
                bufs, trips, toff, n_wg = launches[ph]
                plans[ph].run(bufs, trips, toff, n_wg, stream=stream)
        for _ in range(a.warmup):
            step()
        plans[1].status(stream)
        plans[2].status(stream)
        ev = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(a.steps)]
        torch.cuda.synchronize()
        for i in range(a.steps):
            ev[i][0].record(stream)
            bufs, trips, toff, n_wg = launches[1]
            plans[1].run(bufs, trips, toff, n_wg, stream=stream)
            ev[i][1].record(stream)
            bufs, trips, toff, n_wg = launches[2]
            plans[2].run(bufs, trips, toff, n_wg, stream=stream)
            ev[i][2].record(stream)
        torch.cuda.synchronize()
        plans[1].status(stream)
        plans[2].status(stream)
        p1 = [e[0].elapsed_time(e[1]) for e in ev]
        p2 = [e[1].elapsed_time(e[2]) for e in ev]
        res[name] = {"ms_mean": (sum(p1) + sum(p2)) / a.steps, "phase1_ms": sum(p1) / a.steps,
                     "phase2_ms": sum(p2) / a.steps}
    c = moe.counts.astype(np.float64)
    flop = float(6.0 * c.sum() * H * F)
    # per-expert roofline: every expert's weights and token rows cross HBM once
    f_e = 6.0 * c * H * F
    b_e = np.where(c > 0, 3.0 * H * F * 2, 0.0) + c * (H * 2 + F * 2 * 2 + H * 2)
    t_roof = float(np.sum(np.maximum(f_e / (MFMA_BF16_PEAK_TFLOPS * 1e12), b_e / (HBM_PEAK_GBS * 1e9))))
    bf = res.get("barrier_free", next(iter(res.values())))
    ms = bf["ms_mean"]
    tflops = flop / (ms * 1e-3) / 1e12
    out = {
        "metric": METRIC, "value": tflops, "unit": "TFLOP/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "MoE grouped GEMM, 32768 tokens top-1 to 64 experts (Zipf 1.1 counts), hidden 4096, "
                               "ffn 1408, SiLU-gated, bf16 weights N(0,0.02); gate/up launch + down launch",
                   "tokens": T, "experts": len(c), "hidden": H, "ffn": F,
                   "ring_across_m_tiles": "linearized MMA->LOAD (extension)" if a.moe_ring == "linear"
                   else "ACQL drain (paper's relation)", "parallelism": "single GPU"},
        "latency_us": {kk: v["ms_mean"] * 1e3 for kk, v in res.items()},
        "phase_us": {kk: [v["phase1_ms"] * 1e3, v["phase2_ms"] * 1e3] for kk, v in res.items()},
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / MFMA_BF16_PEAK_TFLOPS, "traffic": None},
        "per_expert_roofline": {"time_us": t_roof * 1e6, "frac": t_roof / (ms * 1e-3)},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    emit(out, a, "moe")


def bench_rmsnorm(a):
    """RMSNorm + per-row FP8 (E4M3) quantization of a 32768 x 8192 bf16
    activation matrix: load / vector / store engines over a software-pipelined
    row loop (x and q rings double-buffered); both synchronization modes.
    HBM roofline: X read once, codes and scales written once."""
    import numpy as np
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import RMS_H, RMS_T, rmsnorm_program, rmsnorm_worklist
    from workloads.tensors import rmsnorm_inputs

    t, h = RMS_T, RMS_H
    nx, nq = (int(v) for v in a.rms_ring.split(","))
    ri = rmsnorm_inputs(seed=a.seed, t=t, h=h)
    X = torch.from_numpy(ri.x.view(np.int16)).cuda()
    G = torch.from_numpy(ri.gamma.view(np.int16)).cuda()
    Q = torch.empty(t * h, dtype=torch.uint8, device="cuda")
    S = torch.empty(t, dtype=torch.float32, device="cuda")
    base_np, tt = rmsnorm_worklist(t, a.rms_wg)
    base = torch.from_numpy(base_np).cuda()
    t_np, o_np = tt.flat()
    trips, toff = torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda()
    res, outs = {}, {}
    for name in a.modes.split(","):
        mode = MODE_BARRIER_FREE if name == "barrier_free" else MODE_BARRIER
        plan = Plan(rmsnorm_program(t, h, a.rms_waves, nx, nq), mode, alloc_of(a, mode))
        res[name] = time_mode(plan, [base, X, G, Q, S], trips, toff, a.rms_wg, a.steps, a.warmup)
        outs[name] = (Q.clone(), S.clone())
    if len(outs) == 2 and not (torch.equal(outs["barrier_free"][0], outs["barrier"][0]) and
                               torch.equal(outs["barrier_free"][1], outs["barrier"][1])):
        raise SystemExit("rmsnorm: the two modes disagree")
    bytes_alg = 2.0 * t * h + 2.0 * h + 1.0 * t * h + 4.0 * t
    bf = res.get("barrier_free", next(iter(res.values())))
    ms = bf["ms_mean"]
    gbs = bytes_alg / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": gbs, "unit": "GB/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "RMSNorm + per-row FP8 E4M3 quantization, X bf16 32768 x 8192 ~ N(0,1) with "
                               "0.5% outlier channels x20, gamma bf16 1 + N(0,0.1); load / vector / store engines",
                   "t": t, "h": h, "n_wg": a.rms_wg, "vector_waves": a.rms_waves, "x_ring": nx, "q_ring": nq,
                   "parallelism": "single GPU"},
        "latency_us": {kk: v["ms_mean"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    if not a.no_cpu_baseline:
        from oracle import mathref
        rows, t0 = 0, time.perf_counter()
        while rows < t and time.perf_counter() - t0 < 10.0:
            mathref.rmsnorm_fp8_rows(ri.x, ri.gamma, 1e-6, range(rows, min(t, rows + 64)))
            rows = min(t, rows + 64)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": rows * (3.0 * h + 4.0) / dt / 1e9, "unit": "GB/s", "cores": 1,
                               "kind": "oracle", "sample": f"first {rows} of {t} rows in {dt:.1f} s"}
    emit(out, a, "rms")


def bench_adamw(a):
    """AdamW step over fp32 parameters (p, g, m, v read, p, m, v written in
    place): load / vector / store engines over a loop of parameter chunks
    with a double-buffered ring; both synchronization modes.  Each mode is
    first run once on a fresh copy of the state and the two results compared;
    the timed launches then keep updating the state in place."""
    import numpy as np
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import ADAM_HP, adamw_program, adamw_worklist
    from workloads.tensors import adamw_inputs

    n, chunk = a.adam_params, a.adam_chunk
    n_chunks = -(-n // chunk)
    n_wg = a.adam_wg or max(1, min(1024, -(-n_chunks // 2)))
    ai = adamw_inputs(seed=a.seed, n=n)
    base_np, tt = adamw_worklist(n, chunk, n_wg)
    base = torch.from_numpy(base_np).cuda()
    t_np, o_np = tt.flat()
    trips, toff = torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda()
    G = torch.from_numpy(ai.g).cuda()
    hp = ADAM_HP
    res, outs = {}, {}
    for name in a.modes.split(","):
        mode = MODE_BARRIER_FREE if name == "barrier_free" else MODE_BARRIER
        plan = Plan(adamw_program(n, chunk, a.adam_waves, a.adam_ring, hp["lr"], hp["b1"], hp["b2"], hp["eps"],
                                  hp["wd"], hp["t"]), mode, alloc_of(a, mode))
        P, M, V = (torch.from_numpy(x.copy()).cuda() for x in (ai.p, ai.m, ai.v))
        plan.run([base, P, G, M, V], trips, toff, n_wg)
        plan.status()
        outs[name] = (P.clone(), M.clone(), V.clone())
        res[name] = time_mode(plan, [base, P, G, M, V], trips, toff, n_wg, a.steps, a.warmup)
    if len(outs) == 2 and not all(torch.equal(x, y) for x, y in zip(outs["barrier_free"], outs["barrier"])):
        raise SystemExit("adamw: the two modes disagree")
    bytes_alg = 28.0 * n
    bf = res.get("barrier_free", next(iter(res.values())))
    ms = bf["ms_mean"]
    gbs = bytes_alg / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": gbs, "unit": "GB/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"AdamW step over {n} fp32 parameters (p ~ N(0,0.02), g ~ N(0,0.01) with 1% x30, "
                               "m, v synthetic state), lr 1e-3, betas (0.9, 0.999), eps 1e-8, wd 0.01, step 10; "
                               "load / vector / store engines",
                   "params": n, "chunk": chunk, "n_wg": n_wg, "vector_waves": a.adam_waves, "ring": a.adam_ring,
                   "parallelism": "single GPU"},
        "latency_us": {kk: v["ms_mean"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    if not a.no_cpu_baseline:
        from oracle import mathref
        done, t0 = 0, time.perf_counter()
        while done < n and time.perf_counter() - t0 < 10.0:
            hi = min(n, done + (1 << 20))
            mathref.adamw_step(ai.p[done:hi], ai.g[done:hi], ai.m[done:hi], ai.v[done:hi], hp["lr"], hp["b1"],
                               hp["b2"], hp["eps"], hp["wd"], hp["t"])
            done = hi
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": 28.0 * done / dt / 1e9, "unit": "GB/s", "cores": 1, "kind": "oracle",
                               "sample": f"{done} of {n} parameters in {dt:.2f} s"}
    emit(out, a, "adamw")


def bench_ring(a):
    """The chain's two engines on a 4-slot ring indexed by the monotone
    register of the inner loop, 1024 workgroups, outer trip 64, inner trips
    U[1, 8], on the interpreter: the paper's form (an ACQ instruction whose
    C3 dependency drains the previous trip's reads at every trip start)
    against one linearized-offset dependency (an extension, not in the
    paper), both barrier-free, and the barrier mode."""
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import ring_workload

    n_wg = 1024
    res, vals = {}, {}
    for name, linear, mode in (("linearized", True, MODE_BARRIER_FREE), ("acq_drain", False, MODE_BARRIER_FREE),
                               ("barrier", False, MODE_BARRIER)):
        w = ring_workload(seed=a.seed, outer=64, inner_max=8, n_wg=n_wg, ring_slots=4, linear=linear)
        t_np, o_np = w.trips.flat()
        trips, toff = torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda()
        base, x = torch.from_numpy(w.base).cuda(), torch.from_numpy(w.x).cuda()
        out = torch.zeros(n_wg * 256, dtype=torch.float32, device="cuda")
        plan = Plan(w.prog, mode)
        res[name] = time_mode(plan, [base, x, out], trips, toff, n_wg, a.steps, a.warmup)
        vals[name] = out.clone()
        inner = w.n_tiles
    if not (torch.equal(vals["linearized"], vals["acq_drain"]) and torch.equal(vals["linearized"], vals["barrier"])):
        raise SystemExit("ring: the forms disagree")
    ms = res["linearized"]["ms_mean"]
    bytes_alg = 256 * 4.0 * inner + n_wg * 256 * 4.0
    gbs = bytes_alg / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC, "value": 2.0 * inner / (ms * 1e-3), "unit": "ops/s", "n_gpus": 1, "steps": a.steps,
        "warmup": a.warmup, "ms_per_step": ms, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "2-engine ring across trips (interpreter): 1024 workgroups, outer 64, inner U[1,8], "
                               "256-fp32 tiles, 4-slot ring indexed by the monotone register",
                   "inner_iterations": inner, "parallelism": "single GPU"},
        "latency_us": {kk: v["ms_mean"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None},
        "speedup_linearized_vs_acq_drain": res["acq_drain"]["ms_mean"] / ms,
        "speedup_vs_barrier": res["barrier"]["ms_mean"] / ms,
    }
    print(json.dumps(out), flush=True)


def bf16_bits_as_f32(bits):
    import numpy as np
    return (bits.astype(np.uint32) << 16).view(np.float32)


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {a.gpus}); the hot path is intra-workgroup "
              "synchronization and is not sharded across GPUs in this build.", file=sys.stderr)
        sys.exit(2)
    import numpy as np
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import stream_workload

    torch.cuda.set_device(0)
    if a.workload == "gemm":
        bench_gemm(a)
        return
    if a.workload == "attn":
        bench_attn(a)
        return
    if a.workload == "moe":
        bench_moe(a)
        return
    if a.workload == "rmsnorm":
        bench_rmsnorm(a)
        return
    if a.workload == "adamw":
        bench_adamw(a)
        return
    if a.workload == "ring":
        bench_ring(a)
        return
    w = stream_workload(seed=a.seed, n_wg=a.n_wg, outer=a.outer, n_gen=a.n_gen)
    trips_np, off_np = w.trips.flat()
    trips = torch.from_numpy(trips_np).cuda()
    toff = torch.from_numpy(off_np).cuda()
    base = torch.from_numpy(w.base).cuda()
    x = torch.from_numpy(w.x).cuda()
    y = torch.empty(w.n_tiles * 64, dtype=torch.float32, device="cuda")
    inner = int(w.counts.sum())
    ops = 3 * inner
    bytes_alg = 2 * 64 * 4 * inner                  # each tile read once and written once
    res = {}
    modes = a.modes.split(",")
    for name in modes:
        mode = MODE_BARRIER_FREE if name == "barrier_free" else MODE_BARRIER
        plan = Plan(w.prog, mode, alloc_of(a, mode))
        if mode == MODE_BARRIER_FREE:
            resources = plan.stats()
        res[name] = time_mode(plan, [base, x, y], trips, toff, a.n_wg, a.steps, a.warmup)
        ok = torch.equal(y, x.reshape(-1) + 1.0)
        if not ok:
            raise SystemExit(f"{name}: output mismatch")
    bf = res.get("barrier_free", next(iter(res.values())))
    ms = bf["ms_mean"]
    achieved = bytes_alg / (ms * 1e-3) / 1e9
    out = {
        "metric": METRIC,
        "value": ops / (ms * 1e-3),
        "unit": "ops/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "sync-bound stream: load/add/store engines, nest 256 x U[1,16] x U[1,4], "
                               "64-fp32 tiles, 1024 workgroups, one in-place LDS ring",
                   "n_wg": a.n_wg, "outer": a.outer, "innermost_iterations": inner,
                   "ring_generations": a.n_gen, "seed": a.seed, "alloc": a.alloc, "parallelism": "single GPU"},
        "latency_us": {k: v["ms_mean"] * 1e3 for k, v in res.items()},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
        out["barrier_ops_per_s"] = ops / (res["barrier"]["ms_mean"] * 1e-3)
    if "barrier_free" in res:
        out["resources"] = resources
    if not a.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w)
    emit(out, a, "stream3")


if __name__ == "__main__":
    main()
