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
and speedup, the barrier-free latency with the per-instance loop (the
schedule the barrier mode runs, so that only the synchronization differs),
the HBM roofline of the stream kernel, the CPU oracle timed on the host
(single-threaded and on all cores) and, as context, the paper's normalized
latency for its matching kernel (Trainium 2 figures).

Other workloads (--workload): chain (the two-engine chain on one
workgroup), gemm, attn, moe, rmsnorm, adamw, ring; each prints one JSON line
of the same form.
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

# The paper's end-to-end latencies of the barrier-free method normalized to
# its barrier-based baseline (= 1.00) for the kernel matching each workload
# (Section 8.2, Table alloc-sema-combined; AWS Trainium 2): context for the
# ratio measured here, not a target.
PAPER_BF_OVER_BB = {
    "stream": ("AddManyLoop (10^4-iteration element-wise add)", 0.30),
    "gemm": ("TiledMatmul 2048^3", 0.90),
    "gemm_k_unrolled": ("TiledMatmul 2048^3, K-unrolled", 0.55),
    "attn": ("FlashAttention 8192^2 x 128", 0.86),
    "moe": ("Dropless MoE T=2048, E=8, top-2 (0.87-0.88 over its three sizes)", 0.88),
    "rmsnorm": ("RMSNorm + FP8 quantization 32768 x 8192", 0.57),
    "adamw": ("AdamW, 1M parameters", 0.74),
}


def paper_context(workload, res):
    """The measured barrier-free / barrier latency ratio next to the paper's
    for the matching kernel (None when the paper has no counterpart)."""
    if workload not in PAPER_BF_OVER_BB or "barrier" not in res or "barrier_free" not in res:
        return None
    name, ratio = PAPER_BF_OVER_BB[workload]
    return {"paper_kernel": name, "paper_bf_over_bb": ratio, "hardware": "AWS Trainium 2",
            "measured_bf_over_bb": res["barrier_free"]["ms_mean"] / res["barrier"]["ms_mean"]}


def host_info():
    """Host cores and CPU model (the fields lscpu reports)."""
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"nproc": len(os.sched_getaffinity(0)), "cpu_count": os.cpu_count(), "cpu_model": model}


# Oracle work shared with forked worker processes (set before the fork).
_ORACLE_WORK = {}


def _one_blas_thread():
    from threadpoolctl import threadpool_limits
    threadpool_limits(1)


def _oracle_chunk(i):
    """Runs chunk i of the oracle sample registered in _ORACLE_WORK."""
    return _ORACLE_WORK["fn"](_ORACLE_WORK["chunks"][i])


def oracle_rate(fn, chunks, units, budget_s=8.0, max_cores=16):
    """The oracle timed on a bounded sample of the workload: fn(chunk) over
    the chunks in order, first single-threaded (BLAS limited to one thread)
    for about budget_s, then on all host cores (at most max_cores forked
    worker processes, one BLAS thread each) over the following chunks for
    about budget_s of wall time.  units(chunk) is the chunk's work in the
    metric's unit.  Must run before the process initializes the GPU (the
    workers are forked)."""
    import multiprocessing as mp
    from threadpoolctl import threadpool_limits
    cores = max(1, min(max_cores, len(os.sched_getaffinity(0))))
    done, u1, t1 = 0, 0.0, 0.0
    with threadpool_limits(1):
        while done < len(chunks) and t1 < budget_s:
            t0 = time.perf_counter()
            fn(chunks[done])
            t1 += time.perf_counter() - t0
            u1 += units(chunks[done])
            done += 1
    out = {"single_thread_value": u1 / t1, "single_thread_sample": f"{done} chunks in {t1:.1f} s"}
    per_chunk = t1 / max(done, 1)
    want = max(cores, int(budget_s / per_chunk) * cores)
    rest = list(range(done, min(len(chunks), done + want)))
    if len(rest) >= cores and cores > 1:
        _ORACLE_WORK["fn"], _ORACLE_WORK["chunks"] = fn, chunks
        ctx = mp.get_context("fork")
        with ctx.Pool(cores, initializer=_one_blas_thread) as pool:
            t0 = time.perf_counter()
            pool.map(_oracle_chunk, rest, chunksize=1)
            tp = time.perf_counter() - t0
        out["value"] = sum(units(chunks[i]) for i in rest) / tp
        out["cores"] = cores
        out["all_cores_sample"] = f"{len(rest)} chunks in {tp:.1f} s on {cores} processes"
    else:
        out["value"] = out["single_thread_value"]
        out["cores"] = 1
    out["host"] = host_info()
    return out


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--n-wg", type=int, default=1024)
    ap.add_argument("--outer", type=int, default=256)
    ap.add_argument("--n-gen", type=int, default=32)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-measured-peak", action="store_true",
                    help="skip the copy / library-matmul measurement of achievable peaks")
    ap.add_argument("--modes", default="",
                    help="comma-separated modes to time (default: barrier_free,barrier; the stream adds "
                         "barrier_free_per_instance)")
    ap.add_argument("--algorithmic-bytes", action="store_true",
                    help="print the workload's algorithmic HBM bytes per step and exit (no GPU)")

    ap.add_argument("--k-unroll", type=int, default=0, choices=[0, 1, 2, 4, 8],
                    help="GEMM: K steps per copy of the loop bodies (static-trip unrolling)")
    ap.add_argument("--k-unrolled", action="store_true",
                    help="GEMM: the K-unrolled program (K loop removed, 128 steps in straight line, every K-phase "
                         "wait a static immediate), the paper's K-unrolled tiled matmul")
    ap.add_argument("--alloc", default="per_loop", choices=["per_loop", "per_instr"],
                    help="counter allocation of the barrier-free plans (Eq. 5 per loop and engine, "
                         "or Eq. 3 one counter per producer instruction)")
    ap.add_argument("--workload", default="stream",
                    choices=["stream", "chain", "gemm", "attn", "moe", "rmsnorm", "adamw", "ring"],
                    help="stream: the sync-bound microbenchmark (headline); chain: the two-engine chain on one "
                         "workgroup; gemm: 4096^3 bf16 GEMM + bias + GELU; "
                         "attn: varlen attention forward; moe: MoE grouped GEMM; rmsnorm: RMSNorm + FP8 "
                         "quantization of 32768 x 8192 bf16; adamw: AdamW step over fp32 parameters; ring: "
                         "a ring indexed across trips on the interpreter, drained by an ACQ at every trip start "
                         "(the paper's form) vs one linearized-offset dependency (an extension)")
    ap.add_argument("--adam-params", type=int, default=1 << 20, help="adamw: parameters (the paper's 2^20 by default)")
    ap.add_argument("--adam-wg", type=int, default=0, help="adamw: workgroups (0: one per 2 chunks, at most 1024)")
    ap.add_argument("--adam-chunk", type=int, default=1024, help="adamw: parameters per chunk (256, 512, 1024)")
    ap.add_argument("--adam-waves", type=int, default=2, help="adamw: vector-engine waves")
    ap.add_argument("--adam-ring", type=int, default=2, help="adamw: ring slots")
    ap.add_argument("--moe-bm", type=int, default=0, choices=[0, 128, 256],
                    help="moe: token rows per M-tile (0: the library default)")
    ap.add_argument("--moe-mchunk", type=int, default=0,
                    help="moe: at most this many M-tiles per workgroup (0: the default for the tile height)")
    ap.add_argument("--rms-wg", type=int, default=768, help="rmsnorm: workgroups (3 per CU)")
    ap.add_argument("--rms-waves", type=int, default=4, help="rmsnorm: vector-engine waves sharing each row")
    ap.add_argument("--rms-ring", default="2,2", help="rmsnorm: x-ring and q-ring slots")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="after the timed region, run one plain device copy of this many MiB "
                         "(reference dispatch for HBM traffic counters)")
    a = ap.parse_args()
    if not a.modes:
        a.modes = {"stream": "barrier_free,barrier,barrier_free_per_instance",
                   "attn": "barrier_free,barrier_free_linearized,barrier",
                   "moe": "barrier_free,barrier_free_linearized,barrier"}.get(a.workload, "barrier_free,barrier")
    return a


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


def cpu_baseline(w, budget_s=8.0):
    """The CPU oracle's sequential program-order execution of the stream
    workload (fp64 values), on chunks of 16 workgroups: single-threaded, then
    on all host cores (forked before the GPU is initialized)."""
    from oracle import core
    trips, off = w.trips.flat()
    n_wg = w.trips.n_wg

    def run(r):
        lo, hi = r
        base = w.base[lo:hi] - w.base[lo]
        n_t = int(w.counts[lo:hi].sum())
        core.values(w.prog, trips, off[lo:hi], base, w.x[w.base[lo]:w.base[lo] + n_t], n_t * 64)

    chunks = [(lo, min(n_wg, lo + 16)) for lo in range(0, n_wg, 16)]
    # the sample: the whole workload many times over (each chunk is cheap)
    res = oracle_rate(run, chunks * 40, lambda r: 3.0 * float(w.counts[r[0]:r[1]].sum()), budget_s=budget_s)
    res.update(unit="ops/s", kind="oracle",
               sample=f"chunks of 16 of the {n_wg} workgroups, sequential program order in fp64")
    return res


MFMA_BF16_PEAK_TFLOPS = 2500.0


def bench_gemm(a):
    """4096^3 bf16 GEMM + bias + GELU, one 256 x 256 tile per workgroup,
    load / MFMA / epilogue engines; both synchronization modes."""
    import numpy as np
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import GEMM_BK, GEMM_RING, gemm_program, gemm_program_k_unrolled, gemm_trips, gemm_trips_k_unrolled
    from workloads.tensors import gemm_inputs

    m = n = k = 4096
    gi = gemm_inputs(seed=a.seed, m=m, n=n, k=k)
    cpu = None
    if not a.no_cpu_baseline:
        from oracle import mathref
        rows = [np.arange(r, r + 32) for r in range(0, m, 32)] * 4
        cpu = oracle_rate(lambda rr: mathref.gemm_bias_gelu(gi.a[rr], gi.bt, gi.bias), rows,
                          lambda rr: 2.0 * len(rr) * n * k / 1e12)
        cpu.update(unit="TFLOP/s", kind="oracle",
                   sample="output rows in blocks of 32 (fp64 product of the bf16 inputs, bias, exact-erf GELU)")
    torch.cuda.set_device(0)
    dev = lambda bits: torch.from_numpy(bits.view(np.int16)).cuda()
    A, Bt = dev(gi.a), dev(gi.bt)
    bias = torch.from_numpy(gi.bias).cuda()
    C = torch.empty(m * n, dtype=torch.int16, device="cuda")
    tt = gemm_trips_k_unrolled(m, n) if a.k_unrolled else gemm_trips(m, n, k)
    prog = gemm_program_k_unrolled(m, n, k) if a.k_unrolled else gemm_program(m, n, k)
    t_np, o_np = tt.flat()
    trips, toff = torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda()
    res, outs = {}, {}
    for name in a.modes.split(","):
        mode = MODE_BARRIER_FREE if name == "barrier_free" else MODE_BARRIER
        plan = Plan(prog, mode, alloc_of(a, mode))
        C.fill_(-1)
        res[name] = time_mode(plan, [A, Bt, bias, C], trips, toff, tt.n_wg, a.steps, a.warmup,
                              k_unroll=a.k_unroll)
        outs[name] = C.clone()
    if len(outs) == 2 and not torch.equal(outs["barrier_free"], outs["barrier"]):
        raise SystemExit("gemm: the two modes disagree")
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
                   "k_unroll": a.k_unroll or 1, "k_unrolled_program": bool(a.k_unrolled),
                   "parallelism": "single GPU"},
        "latency_us": {kk: v["ms_mean"] * 1e3 for kk, v in res.items()},
        "latency_median_us": {kk: v["ms_median"] * 1e3 for kk, v in res.items()},
        "latency_min_us": {kk: v["ms_min"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / MFMA_BF16_PEAK_TFLOPS, "traffic": None},
        "library_matmul_tflops": flop / (lib_ms * 1e-3) / 1e12,
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    out["paper_context"] = paper_context("gemm_k_unrolled" if a.k_unrolled else "gemm", res)
    if cpu is not None:
        out["cpu_baseline"] = cpu
    emit(out, a, "gemm")


def bench_attn(a):
    """Variable-length attention forward: 32 sequences of U[128, 4096] tokens,
    16 heads of 128; 256 workgroups (one per compute unit) each run a list of
    (sequence, head, 128-query tile) tiles; both synchronization modes."""
    import numpy as np
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import attn_program, attn_worklist
    from workloads.configs import ATTN_NK, ATTN_NV, ATTN_SP
    from workloads.tensors import attn_inputs

    heads = 16
    ai = attn_inputs(seed=a.seed, heads=heads)
    wl = attn_worklist(ai.lengths, heads)
    cpu = None
    if not a.no_cpu_baseline:
        from oracle import mathref
        rng = np.random.default_rng(1)
        items = [(int(b), int(rng.integers(0, heads)), int(rng.integers(0, ai.lengths[b])))
                 for b in rng.integers(0, len(ai.lengths), size=64 * 4096)]
        chunks = [items[i:i + 64] for i in range(0, len(items), 64)]
        scale = 1.0 / np.sqrt(128.0)
        cpu = oracle_rate(lambda it: mathref.attention_rows(ai.q, ai.k, ai.v, ai.cu_seqlens, scale, it), chunks,
                          lambda it: sum(4.0 * 128 * int(ai.lengths[b]) for b, _, _ in it) / 1e12)
        cpu.update(unit="TFLOP/s", kind="oracle",
                   sample="output rows of random (sequence, head, query row) items in blocks of 64 "
                          "(fp64 softmax attention over the whole sequence)")
    torch.cuda.set_device(0)
    dev = lambda bits: torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()
    q, k, v = dev(ai.q), dev(ai.k), dev(ai.v)
    o = torch.empty(ai.q.shape, dtype=torch.int16, device="cuda")
    work = torch.from_numpy(wl.work.reshape(-1)).cuda()
    t_np, o_np = wl.trips.flat()
    trips, toff = torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda()
    res, outs = {}, {}
    # barrier_free: the benchmark form (per-trip reuse dependencies and
    # acquire instructions at each tile: the paper's relation only);
    # barrier_free_linearized: the reuse read with the linearized offset
    # across tiles (an extension)
    for name in a.modes.split(","):
        mode = MODE_BARRIER_FREE if name.startswith("barrier_free") else MODE_BARRIER
        prog = attn_program(heads, linear=name == "barrier_free_linearized")
        plan = Plan(prog, mode, alloc_of(a, mode))
        o.fill_(-1)
        res[name] = time_mode(plan, [work, q, k, v, o], trips, toff, wl.trips.n_wg, a.steps, a.warmup)
        outs[name] = o.clone()
    for name in outs:
        if not torch.equal(outs[name], next(iter(outs.values()))):
            raise SystemExit(f"attn: {name} disagrees with the other modes")
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
                   "rings": {"k": ATTN_NK, "v": ATTN_NV, "s_p": ATTN_SP},
                   "ring_across_tiles": "barrier_free: acquires at each tile (the paper's relation); "
                                        "barrier_free_linearized: linearized reuse dependencies (extension)",
                   "parallelism": "single GPU"},
        "latency_us": {kk: v["ms_mean"] * 1e3 for kk, v in res.items()},
        "latency_median_us": {kk: v["ms_median"] * 1e3 for kk, v in res.items()},
        "latency_min_us": {kk: v["ms_min"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / MFMA_BF16_PEAK_TFLOPS, "traffic": None},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    if "barrier" in res and "barrier_free_linearized" in res:
        out["speedup_vs_barrier_linearized"] = res["barrier"]["ms_mean"] / res["barrier_free_linearized"]["ms_mean"]
    out["paper_context"] = paper_context("attn", res)
    if cpu is not None:
        out["cpu_baseline"] = cpu
    emit(out, a, "attn")


def bench_moe(a):
    """MoE grouped GEMM: 32768 tokens routed top-1 to 64 experts with Zipf(1.1)
    counts, hidden 4096, ffn 1408, SiLU-gated; one step = the gate/up launch
    plus the down launch; both synchronization modes."""
    import numpy as np
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import moe_program, moe_worklist
    from workloads.configs import MOE_BM, MOE_MCHUNKS, MOE_RINGS
    from workloads.tensors import moe_inputs, moe_weights_all

    moe = moe_inputs(seed=a.seed)
    H, F = moe.hidden, moe.ffn
    bm = a.moe_bm or MOE_BM
    mchunk = a.moe_mchunk or MOE_MCHUNKS[bm]
    cpu = None
    if not a.no_cpu_baseline:
        from oracle import mathref
        # blocks of 32 tokens of one expert each (an expert's weights are
        # converted once per block), experts in turn
        chunks = []
        for j in range(64):
            for e in range(len(moe.counts)):
                grp = moe.perm[int(moe.expert_off[e]):int(moe.expert_off[e + 1])]
                if len(grp) >= 32 * (j + 1):
                    chunks.append(grp[32 * j:32 * (j + 1)].tolist())
        cpu = oracle_rate(lambda toks: mathref.moe_tokens(moe, toks), chunks,
                          lambda toks: 6.0 * len(toks) * H * F / 1e12)
        cpu.update(unit="TFLOP/s", kind="oracle",
                   sample="output rows of blocks of 32 tokens of one expert (fp64 gated MLP under the routed expert)")
    torch.cuda.set_device(0)
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
        wl = moe_worklist(moe.counts, ph, H, F, bm=bm, mchunk=mchunk)
        t_np, o_np = wl.trips.flat()
        work = torch.from_numpy(wl.work.reshape(-1)).cuda()
        bufs = [work, perm, eoff, x, wg, wu, h] if ph == 1 else [work, perm, eoff, h, wd, y]
        launches[ph] = (bufs, torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda(), wl.trips.n_wg)
    stream = torch.cuda.current_stream()
    res, outs = {}, {}
    # barrier_free: the paper's relation (ACQL drains the ring at every
    # M-tile); barrier_free_linearized: MMA->LOAD read with the linearized
    # offset across M-tiles (an extension)
    for name in a.modes.split(","):
        mode = MODE_BARRIER_FREE if name.startswith("barrier_free") else MODE_BARRIER
        plans = {ph: Plan(moe_program(ph, H, F, linear=name == "barrier_free_linearized", bm=bm), mode,
                          alloc_of(a, mode))
                 for ph in (1, 2)}
        h.fill_(-1)
        y.fill_(-1)

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
        tot = sorted(x + y for x, y in zip(p1, p2))
        res[name] = {"ms_mean": (sum(p1) + sum(p2)) / a.steps, "phase1_ms": sum(p1) / a.steps,
                     "phase2_ms": sum(p2) / a.steps, "ms_median": tot[len(tot) // 2], "ms_min": tot[0]}
        outs[name] = (h.clone(), y.clone())
    first = next(iter(outs.values()))
    for name, o in outs.items():
        if not all(torch.equal(u, v) for u, v in zip(o, first)):
            raise SystemExit(f"moe: {name} disagrees with the other modes")
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
                   "ring_across_m_tiles": "barrier_free: ACQL drain (paper's relation); "
                                          "barrier_free_linearized: linearized MMA->LOAD (extension)",
                   "m_tile_rows": bm, "m_tiles_per_workgroup_run": mchunk,
                   "ring_slots": [MOE_RINGS[bm, 1][0], MOE_RINGS[bm, 2][0]],
                   "epilogue_slots": [MOE_RINGS[bm, 1][1], MOE_RINGS[bm, 2][1]],
                   "epilogue_slots_note": "0: each chunk of an M-tile in its own 16 KiB of the ring", "n_wg": [launches[1][3], launches[2][3]], "parallelism": "single GPU"},
        "latency_us": {kk: v["ms_mean"] * 1e3 for kk, v in res.items()},
        "latency_median_us": {kk: v["ms_median"] * 1e3 for kk, v in res.items()},
        "latency_min_us": {kk: v["ms_min"] * 1e3 for kk, v in res.items()},
        "phase_us": {kk: [v["phase1_ms"] * 1e3, v["phase2_ms"] * 1e3] for kk, v in res.items()},
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / MFMA_BF16_PEAK_TFLOPS, "traffic": None},
        "per_expert_roofline": {"time_us": t_roof * 1e6, "frac": t_roof / (ms * 1e-3)},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    if "barrier" in res and "barrier_free_linearized" in res:
        out["speedup_vs_barrier_linearized"] = res["barrier"]["ms_mean"] / res["barrier_free_linearized"]["ms_mean"]
    out["paper_context"] = paper_context("moe", res)
    if cpu is not None:
        out["cpu_baseline"] = cpu
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
        "latency_median_us": {kk: v["ms_median"] * 1e3 for kk, v in res.items()},
        "latency_min_us": {kk: v["ms_min"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    out["paper_context"] = paper_context("rmsnorm", res)
    if not a.no_cpu_baseline:
        from oracle import mathref
        rows, t0 = 0, time.perf_counter()
        while rows < t and time.perf_counter() - t0 < 10.0:
            mathref.rmsnorm_fp8_rows(ri.x, ri.gamma, 1e-6, range(rows, min(t, rows + 64)))
            rows = min(t, rows + 64)
        dt = time.perf_counter() - t0
        out["cpu_baseline"] = {"value": rows * (3.0 * h + 4.0) / dt / 1e9, "unit": "GB/s", "cores": 1,
                               "kind": "oracle", "sample": f"first {rows} of {t} rows in {dt:.1f} s",
                               "host": host_info()}
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
    from workloads import ADAM_HP, adamw_default_wg, adamw_program, adamw_worklist
    from workloads.tensors import adamw_inputs

    n, chunk = a.adam_params, a.adam_chunk
    n_chunks = -(-n // chunk)
    n_wg = a.adam_wg or adamw_default_wg(n, chunk)
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
        "latency_median_us": {kk: v["ms_median"] * 1e3 for kk, v in res.items()},
        "latency_min_us": {kk: v["ms_min"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
    out["paper_context"] = paper_context("adamw", res)
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
                               "sample": f"{done} of {n} parameters in {dt:.2f} s", "host": host_info()}
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
        "latency_median_us": {kk: v["ms_median"] * 1e3 for kk, v in res.items()},
        "latency_min_us": {kk: v["ms_min"] * 1e3 for kk, v in res.items()},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None},
        "speedup_linearized_vs_acq_drain": res["acq_drain"]["ms_mean"] / ms,
        "speedup_vs_barrier": res["barrier"]["ms_mean"] / ms,
    }
    print(json.dumps(out), flush=True)


def algorithmic_bytes(a):
    """HBM bytes per step that each workload must move at least (inputs read
    once, outputs written once)."""
    from workloads import chain_workload, ring_workload, stream_workload
    from workloads.configs import RMS_H, RMS_T
    wl = a.workload
    if wl == "stream":
        w = stream_workload(seed=a.seed, n_wg=a.n_wg, outer=a.outer, n_gen=a.n_gen, with_data=False)
        return 512.0 * float(w.counts.sum())                  # 64 fp32 read + 64 fp32 written per iteration
    if wl == "gemm":
        m = n = k = 4096
        return 2.0 * m * k + 2.0 * n * k + 2.0 * m * n + 4.0 * n  # A, B, C bf16 and the fp32 bias
    if wl == "attn":
        from workloads.tensors import attn_lengths
        return 4.0 * float(attn_lengths(seed=a.seed).sum()) * 16 * 128 * 2   # Q, K, V read, O written
    if wl == "moe":
        from workloads.tensors import zipf_counts
        t, e, hid, ffn = 32768, 64, 4096, 1408
        assert int(zipf_counts(t, e, 1.1).sum()) == t
        # every expert's weights, x read, h written and read back, y written
        return 3.0 * e * hid * ffn * 2 + t * hid * 2 + 2.0 * t * ffn * 2 + t * hid * 2
    if wl == "rmsnorm":
        return RMS_T * (3.0 * RMS_H + 4) + 2.0 * RMS_H          # X read, codes + scales written, gamma read
    if wl == "adamw":
        return 28.0 * a.adam_params                             # p, g, m, v read; p, m, v written
    if wl == "chain":
        return sum(1024.0 * chain_workload(seed=sd).n_tiles + 1024.0 for sd in (0, 1, 2)) / 3.0
    if wl == "ring":
        w = ring_workload(seed=a.seed, outer=64, inner_max=8, n_wg=1024, ring_slots=4)
        return 1024.0 * w.n_tiles + 1024.0 * 1024
    raise ValueError(wl)


def bench_chain(a):
    """The two-engine chain on one workgroup (loop A of 16 iterations, inner
    trips U[1, 8], 256-fp32 tiles through a 4-slot ring, seeds 0, 1, 2) on
    its own kernel, and on the generic interpreter for comparison.  Latency
    per launch from events on the stream, and the in-kernel time (the
    longest wave's run time from the per-wave statistics of one instrumented
    launch), both modes; ops/s = 2 engine operations per inner iteration /
    latency."""
    import torch
    from paper_2608_13757_amd import ALLOC_PER_ENGINE, MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from workloads import chain_workload

    seeds = (0, 1, 2)
    ws = {(kern, sd): chain_workload(seed=sd, kernel=kern) for kern in ("chain", "interp") for sd in seeds}
    cpu = None
    if not a.no_cpu_baseline:
        from oracle import core

        def run(sd):
            w = ws[("chain", sd)]
            trips, off = w.trips.flat()
            core.values(w.prog, trips, off, w.base, w.x, 256)
        cpu = oracle_rate(run, list(seeds) * 2000, lambda sd: 2.0 * ws[("chain", sd)].n_tiles, budget_s=4.0)
        cpu.update(unit="ops/s", kind="oracle", sample="the three seeds' chains in turn, sequential program order in fp64")
    torch.cuda.set_device(0)
    mean = lambda vals: sum(vals) / len(vals)
    summary = {}
    for kern in ("chain", "interp"):
        per_seed, res_all = {}, {}
        for sd in seeds:
            w = ws[(kern, sd)]
            t_np, o_np = w.trips.flat()
            trips, toff = torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda()
            base, x = torch.from_numpy(w.base).cuda(), torch.from_numpy(w.x).cuda()
            out = torch.empty(256, dtype=torch.float32, device="cuda")
            r, outs = {}, {}
            for name in a.modes.split(","):
                mode = MODE_BARRIER_FREE if name == "barrier_free" else MODE_BARRIER
                plan = Plan(w.prog, mode, alloc_of(a, mode))
                out.fill_(float("nan"))
                r[name] = time_mode(plan, [base, x, out], trips, toff, 1, a.steps, a.warmup)
                outs[name] = out.clone()
                stats = torch.zeros(plan.n_waves * 8, dtype=torch.int64, device="cuda")
                plan.run([base, x, out], trips, toff, 1, stats=stats)
                plan.status()
                r[name]["in_kernel_us"] = float(stats.view(-1, 8)[:, 0].max().item()) * 0.01   # 100 MHz ticks
            if len(outs) == 2 and not torch.equal(outs["barrier_free"], outs["barrier"]):
                raise SystemExit(f"chain ({kern}) seed {sd}: the two modes disagree")
            if kern == "interp" and "barrier_free" in outs:
                # per-engine counters (Section 6.1), which the interpreter runs
                plan = Plan(w.prog, MODE_BARRIER_FREE, ALLOC_PER_ENGINE)
                out.fill_(float("nan"))
                r["barrier_free_per_engine"] = time_mode(plan, [base, x, out], trips, toff, 1, a.steps, a.warmup)
                if not torch.equal(out, outs["barrier_free"]):
                    raise SystemExit(f"chain (interp) seed {sd}: per-engine counters disagree with per-loop")
                stats = torch.zeros(plan.n_waves * 8, dtype=torch.int64, device="cuda")
                plan.run([base, x, out], trips, toff, 1, stats=stats)
                plan.status()
                r["barrier_free_per_engine"]["in_kernel_us"] = float(stats.view(-1, 8)[:, 0].max().item()) * 0.01
            per_seed[sd] = {"inner_iterations": w.n_tiles,
                            "latency_us": {k: v["ms_mean"] * 1e3 for k, v in r.items()},
                            "in_kernel_us": {k: v["in_kernel_us"] for k, v in r.items()}}
            if "barrier" in r and "barrier_free" in r:
                per_seed[sd]["speedup_vs_barrier"] = r["barrier"]["ms_mean"] / r["barrier_free"]["ms_mean"]
                per_seed[sd]["in_kernel_speedup_vs_barrier"] = (r["barrier"]["in_kernel_us"] /
                                                                r["barrier_free"]["in_kernel_us"])
            for k, v in r.items():
                res_all.setdefault(k, []).append(v)
        ms = {k: mean([v["ms_mean"] for v in vs]) for k, vs in res_all.items()}
        ikus = {k: mean([v["in_kernel_us"] for v in vs]) for k, vs in res_all.items()}
        summary[kern] = {"ms": ms, "in_kernel_us": ikus, "per_seed": per_seed}
    inner = mean([ws[("chain", sd)].n_tiles for sd in seeds])
    ms, ikus = summary["chain"]["ms"], summary["chain"]["in_kernel_us"]
    bfk = "barrier_free" if "barrier_free" in ms else next(iter(ms))
    out = {
        "metric": METRIC, "value": 2.0 * inner / (ms[bfk] * 1e-3), "unit": "ops/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": ms[bfk], "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": "2-engine chain, 1 workgroup: outer loop 16, inner trips U[1,8] per seed, "
                               "256-fp32 tiles U[-1,1] through a 4-slot LDS ring, consumer acc += 0.5 tile",
                   "seeds": list(seeds), "n_wg": 1, "kernel": "chain (load wave + vector wave)",
                   "parallelism": "single GPU"},
        "latency_us": {k: v * 1e3 for k, v in ms.items()},
        "in_kernel_us": ikus,
        "in_kernel_ops_per_s": 2.0 * inner / (ikus[bfk] * 1e-6),
        "per_seed": summary["chain"]["per_seed"],
        "interpreter": {"latency_us": {k: v * 1e3 for k, v in summary["interp"]["ms"].items()},
                        "in_kernel_us": summary["interp"]["in_kernel_us"]},
        "roofline": {"bound": "latency", "achieved": None, "peak": None, "unit": None, "frac": None,
                     "traffic": None,
                     "note": "one workgroup moves about 73 KB: the launch is latency- and sync-bound, "
                             "a fraction of HBM or MFMA peak does not apply"},
        "paper_context": None,
    }
    if len(ms) == 2:
        out["speedup_vs_barrier"] = ms["barrier"] / ms["barrier_free"]
        out["in_kernel_speedup_vs_barrier"] = ikus["barrier"] / ikus["barrier_free"]
        im, ik = summary["interp"]["ms"], summary["interp"]["in_kernel_us"]
        out["interpreter"]["speedup_vs_barrier"] = im["barrier"] / im["barrier_free"]
        out["interpreter"]["in_kernel_speedup_vs_barrier"] = ik["barrier"] / ik["barrier_free"]
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


def bf16_bits_as_f32(bits):
    import numpy as np
    return (bits.astype(np.uint32) << 16).view(np.float32)


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {a.gpus}); the hot path is synchronization "
              "inside one workgroup and is not sharded across GPUs.", file=sys.stderr)
        sys.exit(2)
    if a.algorithmic_bytes:
        print(int(algorithmic_bytes(a)))
        return
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
    if a.workload == "chain":
        bench_chain(a)
        return
    bench_stream(a)


def bench_stream(a):
    """The sync-bound microbenchmark (the headline): both modes, and the
    barrier-free mode again on the per-instance loop (the schedule the
    barrier mode runs)."""
    import torch
    from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, Plan
    from paper_2608_13757_amd.bfs import RUN_PER_INSTANCE
    from workloads import stream_workload

    w = stream_workload(seed=a.seed, n_wg=a.n_wg, outer=a.outer, n_gen=a.n_gen)
    cpu = None if a.no_cpu_baseline else cpu_baseline(w)
    torch.cuda.set_device(0)
    trips_np, off_np = w.trips.flat()
    trips = torch.from_numpy(trips_np).cuda()
    toff = torch.from_numpy(off_np).cuda()
    base = torch.from_numpy(w.base).cuda()
    x = torch.from_numpy(w.x).cuda()
    y = torch.empty(w.n_tiles * 64, dtype=torch.float32, device="cuda")
    ref = x.reshape(-1) + 1.0
    inner = int(w.counts.sum())
    ops = 3 * inner
    bytes_alg = 2 * 64 * 4 * inner                  # each tile read once and written once
    res = {}
    modes = a.modes.split(",")
    for name in modes:
        mode = MODE_BARRIER_FREE if name.startswith("barrier_free") else MODE_BARRIER
        flags = RUN_PER_INSTANCE if name == "barrier_free_per_instance" else 0
        plan = Plan(w.prog, mode, alloc_of(a, mode))
        if name == "barrier_free":
            resources = plan.stats()
        y.fill_(float("nan"))
        res[name] = time_mode(plan, [base, x, y], trips, toff, a.n_wg, a.steps, a.warmup, flags=flags)
        if not torch.equal(y, ref):
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
                   "ring_generations": a.n_gen, "seed": a.seed, "alloc": a.alloc,
                   "barrier_free_loop": "batches of up to 4 consecutive instances (timed value); "
                                        "barrier_free_per_instance: one instance at a time, as barrier mode",
                   "parallelism": "single GPU"},
        "latency_us": {k: v["ms_mean"] * 1e3 for k, v in res.items()},
        "latency_median_us": {k: v["ms_median"] * 1e3 for k, v in res.items()},
        "latency_min_us": {k: v["ms_min"] * 1e3 for k, v in res.items()},
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": None},
    }
    if "barrier" in res and "barrier_free" in res:
        out["speedup_vs_barrier"] = res["barrier"]["ms_mean"] / res["barrier_free"]["ms_mean"]
        out["barrier_ops_per_s"] = ops / (res["barrier"]["ms_mean"] * 1e-3)
    if "barrier" in res and "barrier_free_per_instance" in res:
        out["speedup_vs_barrier_same_schedule"] = (res["barrier"]["ms_mean"] /
                                                   res["barrier_free_per_instance"]["ms_mean"])
    if "barrier_free" in res:
        out["resources"] = resources
    out["paper_context"] = paper_context("stream", res)
    if out["paper_context"] is not None and "barrier_free_per_instance" in res:
        out["paper_context"]["measured_bf_over_bb_same_schedule"] = (res["barrier_free_per_instance"]["ms_mean"] /
                                                                     res["barrier"]["ms_mean"])
    if cpu is not None:
        out["cpu_baseline"] = cpu
    emit(out, a, "stream3")


if __name__ == "__main__":
    main()
