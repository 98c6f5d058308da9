"""GPU parity of the synchronization path (interpreter and stream kernels).

Thresholds, counters and indices must match the oracle bit-exactly; the
tile-machine values must match within 1e-5 max-abs (fp32 stages) and the two
synchronization modes must produce bit-identical outputs."""
import copy
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import core  # noqa: E402
from paper_2608_13757_amd import (ALLOC_PER_ENGINE, ALLOC_PER_INSTR, ALLOC_PER_LOOP, MODE_BARRIER, MODE_BARRIER_FREE,  # noqa: E402
                                  BfsError, Plan, bfs)
from paper_2608_13757_amd.bfs import RUN_LOG_BATCHED, RUN_PER_INSTANCE  # noqa: E402
from tests.gpu_util import (compare_batched_log_with_oracle, compare_log_with_oracle, dev, log_records,  # noqa: E402
                            trip_tensors)
from workloads import (chain_workload, random_nest, stream_fixed_trips, stream_program,  # noqa: E402
                       stream_workload, tile_bases)
from workloads.configs import TripTables, draw_trips  # noqa: E402

pytestmark = pytest.mark.gpu

MODES = [("barrier_free", MODE_BARRIER_FREE), ("barrier", MODE_BARRIER)]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bfs.lib()


def _say(*a):
    print(*a, flush=True, file=sys.stderr)


def _run_tile_machine(w, plan, n_out, cap=0):
    trips, toff = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    out = torch.zeros(n_out, dtype=torch.float32, device="cuda")
    log = None
    if cap:
        log = torch.zeros(plan.debug_log_words(w.trips.n_wg, cap), dtype=torch.int32, device="cuda")
    plan.run([base, x, out], trips, toff, w.trips.n_wg, debug_log=log, debug_capacity=cap)
    plan.status()
    return out.cpu().numpy(), (log.cpu().numpy().view(np.uint32) if cap else None)


# ---------------------------------------------------------------------------
# cfg1: two-engine chain on the interpreter
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kernel", ["chain", "interp"])
@pytest.mark.parametrize("seed", [0, 1, 2])
def test_chain_parity(seed, kernel):
    """cfg1 (one workgroup, loop A of 16, inner trips U[1,8]) on the chain
    kernel and on the generic interpreter: values within 1e-5 of the fp64
    oracle, every threshold equal to the oracle's, both modes bit-identical."""
    _say(f"[chain] seed={seed} kernel={kernel}")
    w = chain_workload(seed, kernel=kernel)
    trips, off = w.trips.flat()
    res = core.run(w.prog, trips, off[0], 0, w.base, w.x, 256)
    outs = {}
    for name, mode in MODES:
        plan = Plan(w.prog, mode)
        out, logw = _run_tile_machine(w, plan, 256, cap=512)
        assert np.abs(out - res.out).max() <= 1e-5
        logs = log_records(plan, logw, 1, 512)
        n = compare_log_with_oracle(w.prog, plan, logs, {0: res.recs}, name)
        assert n > 0
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


# ---------------------------------------------------------------------------
# random tiny nests: every threshold the GPU computes equals the brute force
# ---------------------------------------------------------------------------
def _allocatable(prog):
    ok = []
    for d in prog.deps:
        q = copy.deepcopy(prog)
        q.deps = [d]
        try:
            Plan(q)
            ok.append(d)
        except BfsError:
            pass
    return ok


def test_random_nests_interp_thresholds():
    checked = expected = 0
    for seed in range(150):
        prog, tt = random_nest(seed, max_trip=4 if seed % 2 else 3)
        prog.deps = _allocatable(prog)
        if not prog.deps:
            continue
        trips, off = tt.flat()
        res = core.run(prog, trips, off[0], 0)
        for name, mode in MODES:
            plan = Plan(prog, mode)
            if mode == MODE_BARRIER_FREE:
                expected += len(res.recs)
            else:
                same = [w["same_region"] for w in plan.static_waits()]
                expected += sum(1 for r in res.recs if same[int(r["dep"])])
            t_trips, t_off = trip_tensors(tt)
            base = torch.zeros(1, dtype=torch.int64, device="cuda")
            x = torch.zeros(64, dtype=torch.float32, device="cuda")
            out = torch.zeros(64, dtype=torch.float32, device="cuda")
            cap = 256
            log = torch.zeros(plan.debug_log_words(1, cap), dtype=torch.int32, device="cuda")
            plan.run([base, x, out], t_trips, t_off, 1, debug_log=log, debug_capacity=cap)
            plan.status()
            logs = log_records(plan, log.cpu().numpy().view(np.uint32), 1, cap)
            checked += compare_log_with_oracle(prog, plan, logs, {0: res.recs}, name)
    assert checked == expected and checked > 500


# ---------------------------------------------------------------------------
# per-instruction allocation (Section 5.4, Eq. 3): one counter per producer
# instruction, thresholds equal to the Eq. 1 counts
# ---------------------------------------------------------------------------
def test_random_nests_interp_thresholds_per_instr():
    checked = expected = 0
    for seed in range(150):
        prog, tt = random_nest(seed, max_trip=4 if seed % 2 else 3)
        prog.deps = _allocatable(prog)
        if not prog.deps:
            continue
        trips, off = tt.flat()
        res = core.run(prog, trips, off[0], 0)
        plan = Plan(prog, MODE_BARRIER_FREE, ALLOC_PER_INSTR)
        expected += len(res.recs)
        t_trips, t_off = trip_tensors(tt)
        base = torch.zeros(1, dtype=torch.int64, device="cuda")
        x = torch.zeros(64, dtype=torch.float32, device="cuda")
        out = torch.zeros(64, dtype=torch.float32, device="cuda")
        cap = 256
        log = torch.zeros(plan.debug_log_words(1, cap), dtype=torch.int32, device="cuda")
        plan.run([base, x, out], t_trips, t_off, 1, debug_log=log, debug_capacity=cap)
        plan.status()
        logs = log_records(plan, log.cpu().numpy().view(np.uint32), 1, cap)
        checked += compare_log_with_oracle(prog, plan, logs, {0: res.recs}, "per_instr")
    assert checked == expected and checked > 500


# ---------------------------------------------------------------------------
# per-engine allocation (Section 6.1): one counter per producer engine, the
# thresholds equal to the oracle's per-engine counter values
# ---------------------------------------------------------------------------
def test_random_nests_interp_thresholds_per_engine():
    checked = expected = 0
    for seed in range(150):
        prog, tt = random_nest(seed, max_trip=4 if seed % 2 else 3)
        prog.deps = _allocatable(prog)
        if not prog.deps:
            continue
        trips, off = tt.flat()
        res = core.run(prog, trips, off[0], 0)
        plan = Plan(prog, MODE_BARRIER_FREE, ALLOC_PER_ENGINE)
        expected += len(res.recs)
        t_trips, t_off = trip_tensors(tt)
        base = torch.zeros(1, dtype=torch.int64, device="cuda")
        x = torch.zeros(64, dtype=torch.float32, device="cuda")
        out = torch.zeros(64, dtype=torch.float32, device="cuda")
        cap = 256
        log = torch.zeros(plan.debug_log_words(1, cap), dtype=torch.int32, device="cuda")
        plan.run([base, x, out], t_trips, t_off, 1, debug_log=log, debug_capacity=cap)
        plan.status()
        logs = log_records(plan, log.cpu().numpy().view(np.uint32), 1, cap)
        checked += compare_log_with_oracle(prog, plan, logs, {0: res.recs}, "per_engine")
    assert checked == expected and checked > 500


@pytest.mark.parametrize("case", ["chain", "stream_inplace", "stream_two_rings", "ring_linear"])
def test_per_engine_workload_programs_interp(case):
    """The chain, both stream layouts (with the inner reuse dependencies) and
    the ring program with a linearized dependency, on the interpreter with
    per-engine counters: every threshold equals the oracle's per-engine
    counter value, and the values equal those of per-loop counters."""
    from workloads import ring_workload
    if case == "chain":
        w = chain_workload(seed=1, kernel="interp", n_wg=2)
        n_out = 2 * 256
    elif case == "ring_linear":
        w = ring_workload(seed=1, outer=8, n_wg=3, linear=True)
        n_out = 3 * 256
    else:
        w = stream_workload(seed=2, n_wg=4, outer=6, inner_war=True,
                            layout="inplace" if case == "stream_inplace" else "two_rings",
                            n_gen=32 if case == "stream_inplace" else 8)
        w.prog.kernel = "interp"
        n_out = w.n_tiles * 64
    trips, off = w.trips.flat()
    recs = {}
    for g in range(w.trips.n_wg):
        res = core.run(w.prog, trips, off[g], g)
        rr = res.recs.copy()
        for d, lin in enumerate(w.prog.dep_linear or []):
            if lin:
                rr[rr["dep"] == d] = core.linearized_records(w.prog, res, d)
        recs[g] = rr
    _say(f"[per-engine] {case}")
    plan = Plan(w.prog, MODE_BARRIER_FREE, ALLOC_PER_ENGINE)
    out, logw = _run_tile_machine(w, plan, n_out, cap=2048)
    logs = log_records(plan, logw, w.trips.n_wg, 2048)
    assert compare_log_with_oracle(w.prog, plan, logs, recs, "per_engine") > 0
    ref, _ = _run_tile_machine(w, Plan(w.prog), n_out)
    assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))


def test_per_engine_refused_by_fused_families():
    w = stream_workload(seed=0, n_wg=2, outer=3)
    plan = Plan(w.prog, MODE_BARRIER_FREE, ALLOC_PER_ENGINE)
    t = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([t, t, t], t, t, 1)
    assert e.value.status == bfs.E_UNSUPPORTED


@pytest.mark.parametrize("ring,n_wg,outer", [(2, 64, 9), (3, 5, 16), (8, 3, 12), (1, 2, 5)])
def test_chain_kernel_rings_and_workgroups(ring, n_wg, outer):
    """The chain kernel with other ring depths (one slot: no overlap at all)
    and several independent workgroups: values and thresholds against the
    oracle in both modes."""
    w = chain_workload(seed=4, outer=outer, n_wg=n_wg, ring_slots=ring)
    trips, off = w.trips.flat()
    outs = {}
    for name, mode in MODES:
        _say(f"[chain-rings] ring={ring} n_wg={n_wg} mode={name}")
        plan = Plan(w.prog, mode)
        out, logw = _run_tile_machine(w, plan, n_wg * 256, cap=512)
        recs = {}
        for g in range(n_wg):
            res = core.run(w.prog, trips, off[g], g, w.base, w.x, n_wg * 256)
            assert np.abs(out[g * 256:(g + 1) * 256] - res.out[g * 256:(g + 1) * 256]).max() <= 1e-5
            recs[g] = res.recs
        assert compare_log_with_oracle(w.prog, plan, log_records(plan, logw, n_wg, 512), recs, name) > 0
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


@pytest.mark.parametrize("kernel", ["chain", "interp"])
@pytest.mark.parametrize("seed", [0, 1])
def test_chain_per_instr(seed, kernel):
    _say(f"[chain-per-instr] seed={seed} kernel={kernel}")
    w = chain_workload(seed, kernel=kernel)
    trips, off = w.trips.flat()
    res = core.run(w.prog, trips, off[0], 0, w.base, w.x, 256)
    plan = Plan(w.prog, MODE_BARRIER_FREE, ALLOC_PER_INSTR)
    out, logw = _run_tile_machine(w, plan, 256, cap=512)
    assert np.abs(out - res.out).max() <= 1e-5
    assert compare_log_with_oracle(w.prog, plan, log_records(plan, logw, 1, 512), {0: res.recs}, "per_instr") > 0


@pytest.mark.parametrize("layout", ["inplace", "two_rings"])
def test_stream_per_instr(layout):
    """Thresholds of every wait logged on a few workgroups, and the values of
    an uninstrumented launch (the batched engines)."""
    w = stream_workload(seed=7, n_wg=6, outer=12, layout=layout, inner_war=True)
    trips, off = w.trips.flat()
    recs = {g: core.run(w.prog, trips, off[g], g).recs for g in range(w.trips.n_wg)}
    plan = Plan(w.prog, MODE_BARRIER_FREE, ALLOC_PER_INSTR)
    _say(f"[stream-per-instr] {layout} log")
    out, logw = _run_tile_machine(w, plan, w.n_tiles * 64, cap=4096)
    assert np.array_equal(out, w.x.reshape(-1) + np.float32(1.0))
    assert compare_log_with_oracle(w.prog, plan, log_records(plan, logw, w.trips.n_wg, 4096), recs, "per_instr") > 0
    _say(f"[stream-per-instr] {layout} values")
    out, _ = _run_tile_machine(w, plan, w.n_tiles * 64)
    assert np.array_equal(out, w.x.reshape(-1) + np.float32(1.0))


# ---------------------------------------------------------------------------
# cfg2: sync-bound stream kernel
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("inner_war", [False, True])
def test_stream_small_parity_and_thresholds(inner_war):
    w = stream_workload(seed=0, n_wg=6, outer=12, inner_war=inner_war)
    trips, off = w.trips.flat()
    recs = {g: core.run(w.prog, trips, off[g], g).recs for g in range(w.trips.n_wg)}
    ref = w.x.reshape(-1) + np.float32(1.0)          # the same sum rounded to fp32
    ref64 = core.values(w.prog, trips, off, w.base, w.x, w.n_tiles * 64)
    outs = {}
    for name, mode in MODES:
        _say(f"[stream-small] mode={name}")
        plan = Plan(w.prog, mode)
        out, logw = _run_tile_machine(w, plan, w.n_tiles * 64, cap=4096)
        assert np.abs(out.astype(np.float64) - ref64).max() <= 1e-5
        assert np.array_equal(out, ref)
        logs = log_records(plan, logw, w.trips.n_wg, 4096)
        assert compare_log_with_oracle(w.prog, plan, logs, recs, name) > 0
        outs[name] = out
    assert np.array_equal(outs["barrier_free"], outs["barrier"])


def test_stream_interp_cross_check():
    """The generic interpreter runs the same stream program to the same values."""
    w = stream_workload(seed=3, n_wg=3, outer=5)
    p = copy.deepcopy(w.prog)
    p.kernel = "interp"
    _say("[stream-interp]")
    out, _ = _run_tile_machine(w, Plan(p), w.n_tiles * 64)
    assert np.array_equal(out, w.x.reshape(-1) + np.float32(1.0))


def test_stream_full_size_thresholds_sampled_workgroups():
    """Full per-workgroup nest (outer 256) on a few workgroups with the log on."""
    w = stream_workload(seed=1, n_wg=2, outer=256)
    trips, off = w.trips.flat()
    recs = {g: core.run(w.prog, trips, off[g], g).recs for g in range(2)}
    for name, mode in MODES:
        _say(f"[stream-full-log] mode={name}")
        plan = Plan(w.prog, mode)
        cap = 1 << 15
        out, logw = _run_tile_machine(w, plan, w.n_tiles * 64, cap=cap)
        assert np.array_equal(out, w.x.reshape(-1) + np.float32(1.0))
        assert compare_log_with_oracle(w.prog, plan, log_records(plan, logw, 2, cap), recs, name) > 10000


@pytest.mark.parametrize("seed", [0])
def test_stream_full_size_values(seed):
    """The benchmark configuration: 1024 workgroups, 3-level nest 256 x U[1,16] x U[1,4]."""
    _say(f"[stream-full] seed={seed}: generating")
    w = stream_workload(seed=seed)
    trips, toff = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    ref = torch.from_numpy(w.x.reshape(-1)).cuda() + 1.0
    outs = {}
    for name, mode in MODES:
        _say(f"[stream-full] mode={name}")
        plan = Plan(w.prog, mode)
        y = torch.full((w.n_tiles * 64,), float("nan"), dtype=torch.float32, device="cuda")
        plan.run([base, x, y], trips, toff, w.trips.n_wg)
        plan.status()
        assert torch.equal(y, ref)
        outs[name] = y
    assert torch.equal(outs["barrier_free"], outs["barrier"])


def test_stream_batched_path_thresholds_full_size():
    """The timed code path's waits: the benchmark launch (1024 workgroups,
    nest 256 x U[1,16] x U[1,4], seed 0) with the engines on the batched
    loop of uninstrumented launches, logging one entry per batch wait.  On
    sampled workgroups every logged threshold equals the oracle's at the
    logged instance, bit-exact, and covers every instance of its batch; the
    output equals the per-instance launches' (x + 1)."""
    _say("[stream-batched-log] generating")
    w = stream_workload(seed=0)
    trips, off = w.trips.flat()
    sample = [0, 1, 517, 1023]
    recs = {g: core.run(w.prog, trips, off[g], g).recs for g in sample}
    plan = Plan(w.prog, MODE_BARRIER_FREE)
    cap = 4096
    t_trips, t_off = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    y = torch.full((w.n_tiles * 64,), float("nan"), dtype=torch.float32, device="cuda")
    log = torch.zeros(plan.debug_log_words(w.trips.n_wg, cap), dtype=torch.int32, device="cuda")
    _say("[stream-batched-log] run")
    plan.run([base, x, y], t_trips, t_off, w.trips.n_wg, debug_log=log, debug_capacity=cap, flags=RUN_LOG_BATCHED)
    plan.status()
    assert torch.equal(y, torch.from_numpy(w.x.reshape(-1)).cuda() + 1.0)
    words = log.cpu().numpy().view(np.uint32)
    logs = log_records(plan, words, w.trips.n_wg, cap)
    logs = {k: v for k, v in logs.items() if k[0] in sample}
    n = compare_batched_log_with_oracle(w.prog, logs, recs)
    # batches: fewer entries than instances on the inner waits
    n_inner = sum(int((recs[g]["dep"] == 0).sum()) for g in sample)
    n_batched = sum(len(logs.get((g, 0), [])) for g in sample)
    assert n > 0 and n_batched < n_inner


def test_stream_per_instance_flag_values():
    """BFS_RUN_PER_INSTANCE: the barrier-free engines run the per-instance
    loop uninstrumented (the schedule of barrier mode); values equal x + 1 at
    the benchmark shape."""
    w = stream_workload(seed=2, n_wg=256)
    trips, toff = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    y = torch.full((w.n_tiles * 64,), float("nan"), dtype=torch.float32, device="cuda")
    _say("[stream-per-instance]")
    plan = Plan(w.prog, MODE_BARRIER_FREE)
    plan.run([base, x, y], trips, toff, w.trips.n_wg, flags=RUN_PER_INSTANCE)
    plan.status()
    assert torch.equal(y, torch.from_numpy(w.x.reshape(-1)).cuda() + 1.0)


@pytest.mark.parametrize("m_trips,i_trip,ok", [([16] * 8, 4, True), ([16, 17, 16], 4, False), ([3] * 8, 5, False)])
def test_stream_ring_trip_bounds(m_trips, i_trip, ok):
    """Trips at the in-place ring's bounds (M trip n_gen / 2 = 16, I trip
    per_gen = 4) run; one past either bound is reported as invalid input
    (clamped on the device, so the ring never races), in both the batched
    and the per-instance loops; barrier mode has no bound."""
    p = stream_program()
    tt = stream_fixed_trips(p, m_trips, i_trip, n_wg=4)
    base_np, counts = tile_bases(tt, p.loop_id("I"))
    n_tiles = int(counts.sum())
    trips, toff = trip_tensors(tt)
    base = dev(base_np)
    x = torch.rand(n_tiles * 64, dtype=torch.float32, device="cuda")
    for name, mode, flags in (("batched", MODE_BARRIER_FREE, 0), ("per_instance", MODE_BARRIER_FREE, RUN_PER_INSTANCE),
                              ("barrier", MODE_BARRIER, 0)):
        _say(f"[stream-bounds] m={m_trips[:3]} i={i_trip} {name}")
        y = torch.full((n_tiles * 64,), float("nan"), dtype=torch.float32, device="cuda")
        plan = Plan(p, mode)
        plan.run([base, x, y], trips, toff, tt.n_wg, flags=flags)
        if ok or mode == MODE_BARRIER:
            plan.status()
            assert torch.equal(y, x + 1.0)
        else:
            with pytest.raises(BfsError) as e:
                plan.status()
            assert e.value.status == bfs.E_INVALID


# Launches without the debug log run engines specialised on their exact number
# of inner waits: trips of I that fit one generation of slots take the short
# loop, longer trips (slots reused within the trip, ordered by the offset
# per_gen dependencies) the general one; two_rings gives the add engine two
# inner waits.
UNINSTRUMENTED = [("inplace", 4, False), ("inplace", 2, True), ("two_rings", 4, True), ("two_rings", 2, True)]


@pytest.mark.parametrize("layout,per_gen,inner_war", UNINSTRUMENTED)
def test_stream_uninstrumented_values(layout, per_gen, inner_war):
    w = stream_workload(seed=5, n_wg=64, outer=32, inner_war=inner_war, layout=layout)
    w.prog = stream_program(per_gen=per_gen, inner_war=inner_war, layout=layout)
    trips, toff = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    ref = torch.from_numpy(w.x.reshape(-1)).cuda() + 1.0
    for name, mode in MODES:
        _say(f"[stream-uninstr] {layout} per_gen={per_gen} inner_war={inner_war} mode={name}")
        y = torch.full((w.n_tiles * 64,), float("nan"), dtype=torch.float32, device="cuda")
        plan = Plan(w.prog, mode)
        plan.run([base, x, y], trips, toff, w.trips.n_wg)
        plan.status()
        assert torch.equal(y, ref)


@pytest.mark.parametrize("n_gen,mid_max,per_gen", [(2, 1, 4), (4, 2, 4), (6, 3, 4), (6, 3, 2)])
def test_stream_tight_ring_values(n_gen, mid_max, per_gen):
    """The in-place ring at its fewest generations for the M trips (twice the
    largest): the load engine waits for the store engine two O iterations
    back at nearly every O iteration, so it retires the batches it holds
    before blocking, and M-iteration pairs wrap around the ring (six
    generations, trips up to three: a pair can straddle the wrap), also with
    two slots per generation (batches and pairs of at most two).  Outputs
    equal x + 1 in both modes and with the batched waits logged, every
    threshold equals the oracle's."""
    w = stream_workload(seed=11, n_wg=32, outer=64, mid_max=mid_max, inner_max=per_gen, n_gen=n_gen)
    trips, toff = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    ref = torch.from_numpy(w.x.reshape(-1)).cuda() + 1.0
    for name, mode in MODES:
        _say(f"[stream-tight] n_gen={n_gen} mid_max={mid_max} per_gen={per_gen} mode={name}")
        y = torch.full((w.n_tiles * 64,), float("nan"), dtype=torch.float32, device="cuda")
        plan = Plan(w.prog, mode)
        plan.run([base, x, y], trips, toff, w.trips.n_wg)
        plan.status()
        assert torch.equal(y, ref)
    plan = Plan(w.prog, MODE_BARRIER_FREE)
    cap = 4096
    sample = [0, 17, 31]
    log = torch.zeros(plan.debug_log_words(w.trips.n_wg, cap), dtype=torch.int32, device="cuda")
    y = torch.full((w.n_tiles * 64,), float("nan"), dtype=torch.float32, device="cuda")
    plan.run([base, x, y], trips, toff, w.trips.n_wg, debug_log=log, debug_capacity=cap, flags=RUN_LOG_BATCHED)
    plan.status()
    assert torch.equal(y, ref)
    t_all, o_all = w.trips.flat()
    logs = log_records(plan, log.cpu().numpy().view(np.uint32), w.trips.n_wg, cap)
    recs = {g: core.run(w.prog, t_all, o_all[g], g).recs for g in sample}
    logs = {k: v for k, v in logs.items() if k[0] in sample}
    assert compare_batched_log_with_oracle(w.prog, logs, recs) > 0


def test_stream_uninstrumented_watchdog_ends():
    """A one-poll watchdog on the uninstrumented kernel: every engine that
    gives up finishes its trips without waiting, so the launch ends, with the
    deadlock reported or not; the plan runs normally afterwards."""
    w = stream_workload(seed=6, n_wg=64, outer=16)
    plan = Plan(w.prog)
    trips, toff = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    y = torch.zeros(w.n_tiles * 64, dtype=torch.float32, device="cuda")
    _say("[stream-watchdog-uninstr]")
    plan.run([base, x, y], trips, toff, w.trips.n_wg, watchdog_polls=1)
    try:
        plan.status()
    except BfsError as e:
        assert e.status == bfs.E_DEADLOCK
    plan.run([base, x, y], trips, toff, w.trips.n_wg)
    plan.status()
    assert torch.equal(y, torch.from_numpy(w.x.reshape(-1)).cuda() + 1.0)


# ---------------------------------------------------------------------------
# failure handling: an unsatisfiable wait is reported, and the kernel ends
# ---------------------------------------------------------------------------
@pytest.mark.parametrize("kernel", ["interp", "chain", "stream3"])
def test_watchdog_reports_deadlock(kernel):
    _say(f"[watchdog] {kernel}")
    if kernel in ("interp", "chain"):
        w = chain_workload(0, kernel=kernel)
        n_out = 256
    else:
        w = stream_workload(seed=0, n_wg=2, outer=3)
        n_out = w.n_tiles * 64
    plan = Plan(w.prog)
    trips, toff = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    out = torch.zeros(n_out, dtype=torch.float32, device="cuda")
    plan.run([base, x, out], trips, toff, w.trips.n_wg, watchdog_polls=2000, fault_dep=0, fault_delta=1 << 20)
    with pytest.raises(BfsError) as e:
        plan.status()
    assert e.value.status == bfs.E_DEADLOCK
    # the plan is usable again afterwards
    plan.run([base, x, out], trips, toff, w.trips.n_wg)
    plan.status()


def test_stream_program_shape_is_checked():
    p = stream_program()
    p.instrs[p.instr_id("ADD")].opcode = 2
    plan = Plan(p)
    t = torch.zeros(4, dtype=torch.int32, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([t, t, t], t, t, 1)
    assert e.value.status == bfs.E_UNSUPPORTED


def test_random_nests_deeper_all_allocations():
    """Deeper and wider random nests than the tests above (depth up to 4,
    trips up to 5 including empty conditionals, up to 10 dependencies with
    offsets up to 4, 2 to 4 engines), three workgroups with trip tables of
    their own, each program under the per-loop, per-instruction and
    per-engine allocations barrier-free and per-loop in barrier mode: every
    logged threshold of every workgroup equals the oracle's."""
    n_wg = 3
    checked = expected = 0
    base = torch.zeros(n_wg, dtype=torch.int64, device="cuda")
    x = torch.zeros(64, dtype=torch.float32, device="cuda")
    out = torch.zeros(64 * n_wg, dtype=torch.float32, device="cuda")
    cap = 1024
    for seed in range(5000, 6000):
        rng = np.random.default_rng(seed)
        kw = dict(max_depth=int(rng.integers(2, 5)), max_trip=int(rng.integers(1, 6)),
                  n_deps=int(rng.integers(4, 11)), max_k=int(rng.integers(0, 5)), n_engines=int(rng.integers(2, 5)))
        prog0, tt1 = random_nest(seed, **kw)

        def draw(l, n):
            return rng.integers(0, (1 if prog0.loop_is_cond[l] else kw["max_trip"]) + 1, size=n)
        tt = TripTables([tt1.per_wg[0]] + [draw_trips(prog0, draw) for _ in range(n_wg - 1)])
        trips, off = tt.flat()
        t_trips, t_off = trip_tensors(tt)
        for alloc, key in ((ALLOC_PER_LOOP, "barrier_free"), (ALLOC_PER_INSTR, "per_instr"),
                           (ALLOC_PER_ENGINE, "per_engine")):
            prog = copy.deepcopy(prog0)
            ok = []
            for d in prog.deps:
                q = copy.deepcopy(prog)
                q.deps = [d]
                try:
                    Plan(q, MODE_BARRIER_FREE, alloc)
                    ok.append(d)
                except BfsError:
                    pass
            prog.deps = ok
            if not prog.deps:
                continue
            recs = {g: core.run(prog, trips, off[g], g).recs for g in range(n_wg)}
            modes = [(key, MODE_BARRIER_FREE)] + ([("barrier", MODE_BARRIER)] if alloc == ALLOC_PER_LOOP else [])
            for name, mode in modes:
                plan = Plan(prog, mode, alloc if mode == MODE_BARRIER_FREE else ALLOC_PER_LOOP)
                same = [w["same_region"] for w in plan.static_waits()] if mode == MODE_BARRIER else None
                for g in range(n_wg):
                    expected += len(recs[g]) if same is None else sum(1 for r in recs[g] if same[int(r["dep"])])
                log = torch.zeros(plan.debug_log_words(n_wg, cap), dtype=torch.int32, device="cuda")
                plan.run([base, x, out], t_trips, t_off, n_wg, debug_log=log, debug_capacity=cap)
                plan.status()
                logs = log_records(plan, log.cpu().numpy().view(np.uint32), n_wg, cap)
                checked += compare_log_with_oracle(prog, plan, logs, recs, name)
    assert checked == expected and checked > 30000
