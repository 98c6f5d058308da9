"""Barrier fallback for dependencies outside the allocatable cases (Section
5.2, falling back to the barrier scheme of Section 3.4), on the CPU: the
library's classification against the oracle's, the oracle's values for a
pipeline that needs the fallback against their closed form, race coverage
with and without the fallback barriers, and schedule exploration of the
hybrid implementation (semaphores for the allocatable dependencies, drain
barriers for the others)."""
import copy

import numpy as np
import pytest

from oracle import cases, core, hazard
from paper_2608_13757_amd import ALLOC_PER_INSTR, ALLOC_PER_LOOP, KASE_FALLBACK, BfsError, Plan, bfs
from tests.schedule_sim import Model, explore
from workloads import lag_pipeline_workload, random_nest


def _satisfiable(prog):
    q = copy.deepcopy(prog)
    q.deps = [d for j, d in enumerate(prog.deps) if cases.classify(prog, j)[0] != cases.ORDER]
    return q


def _nests(n):
    for seed in range(n):
        prog, tt = random_nest(seed, max_trip=4 if seed % 2 else 3)
        prog = _satisfiable(prog)
        if prog.deps:
            yield seed, prog, tt


def test_classification_matches_oracle():
    """Every satisfiable dependency of 300 random nests: case, S, P and
    direction equal the oracle's; without the flag the planner refuses
    exactly the programs with a fallback dependency."""
    n_fb = n_prog = 0
    for seed, prog, _ in _nests(300):
        plan = Plan(prog, fallback=True)
        want = [cases.classify(prog, d) for d in range(len(prog.deps))]
        for f, (case, S, P, fwd) in zip(plan.formulas(), want):
            assert (f["kase"], f["loop_S"], f["loop_P"], bool(f["forward"])) == (case, S, P, fwd), (seed, f)
            if case == cases.FALLBACK:
                assert f["counter"] == -1
                for r, h in ((1, 1), (5, 3), (9, 9)):
                    assert plan.eval_threshold(f["dep"], r, h) == 0
        has_fb = any(c == cases.FALLBACK for c, *_ in want)
        st = plan.stats()
        assert st["n_fallback"] == sum(c == cases.FALLBACK for c, *_ in want)
        assert st["n_sync_points"] == len(cases.barrier_loops(prog))
        assert st["n_waits"] == len(prog.deps) - st["n_fallback"]
        if has_fb:
            with pytest.raises(BfsError) as e:
                Plan(prog)
            assert e.value.status == bfs.E_NOT_ALLOCATABLE
            n_fb += 1
        else:
            Plan(prog)
        n_prog += 1
    assert n_fb > 60 and n_prog - n_fb > 60


def test_unknown_plan_flags_rejected():
    w = lag_pipeline_workload()
    p = Plan(w.prog, fallback=True)
    lib = bfs.lib()
    import ctypes as C
    h = C.c_void_p()
    assert lib.bfs_plan_create(C.addressof(p._prog), 0, 0, 2, C.byref(h)) == bfs.E_INVALID


@pytest.mark.parametrize("lag,ring", [(2, 3), (3, 5), (1, 2), (2, 6)])
def test_lag_pipeline_oracle_closed_form(lag, ring):
    """The oracle's output of the pipeline equals 0.5 times the sum of the
    workgroup's first trip(O) - lag tiles (none when O runs lag times or
    fewer)."""
    w = lag_pipeline_workload(seed=lag + ring, n_wg=6, outer_min=1, outer_max=12, lag=lag, ring_slots=ring)
    trips, off = w.trips.flat()
    vals = core.values(w.prog, trips, off, w.base, w.x, w.trips.n_wg * 256).reshape(-1, 256)
    O = w.prog.loop_id("O")
    for wg in range(w.trips.n_wg):
        T, b = int(w.trips.per_wg[wg][O][0]), int(w.base[wg])
        ref = 0.5 * w.x[b:b + max(T - lag, 0)].astype(np.float64).sum(0)
        assert np.array_equal(vals[wg], ref), wg


@pytest.mark.parametrize("lag,ring", [(2, 3), (3, 5), (1, 2)])
def test_lag_pipeline_race_coverage(lag, ring):
    """With a barrier at the end of every O iteration the conflicting
    accesses are ordered; with the fallback dependencies waiting for nothing
    and no barrier, the ring slot reuse races."""
    w = lag_pipeline_workload(seed=1, n_wg=1, outer_min=10, outer_max=10, lag=lag, ring_slots=ring)
    prog = w.prog
    trips, off = w.trips.flat()
    res = core.run(prog, trips, off[0], 0, base=w.base, x=w.x, out_len=256)
    loops = cases.barrier_loops(prog)
    assert loops == {prog.loop_id("O")}
    assert hazard.check(prog, res, "barrier_free", barrier_loops=loops) == []
    fb = [d for d in range(len(prog.deps)) if cases.classify(prog, d)[0] == cases.FALLBACK]
    thr = np.array([0 if int(r["dep"]) in fb else int(r["sem_thr"]) for r in res.recs])
    assert hazard.check(prog, res, "barrier_free", thresholds=thr, barrier_loops=loops) == []
    assert hazard.check(prog, res, "barrier_free", thresholds=thr) != []


def _model(prog, tt, per_instr, **kw):
    plan = Plan(prog, alloc=ALLOC_PER_INSTR if per_instr else ALLOC_PER_LOOP, fallback=True)
    trips, off = tt.flat()
    return Model(prog, plan, trips, off[0], per_instr=per_instr, **kw)


def test_random_nests_hybrid_schedules():
    """Random nests with fallback dependencies, both allocations, 3
    schedules each: the allocatable waits fire exactly when their dependency
    is met, no instance passes its barriers before a fallback dependency is
    met, and no schedule deadlocks."""
    programs = 0
    for seed, prog, tt in _nests(160):
        if not any(cases.classify(prog, d)[0] == cases.FALLBACK for d in range(len(prog.deps))):
            continue
        for per_instr in (False, True):
            m = _model(prog, tt, per_instr)
            for s in range(3):
                out = explore(m, 1000 * seed + s, issue_bias=(0.3, 0.7, 0.95)[s])
                assert out.ok, (seed, per_instr, s, out)
        programs += 1
    assert programs > 40


@pytest.mark.parametrize("lag,ring", [(2, 3), (3, 5), (1, 2)])
@pytest.mark.parametrize("per_instr", [False, True])
def test_lag_pipeline_schedules_values(lag, ring, per_instr):
    w = lag_pipeline_workload(seed=2, n_wg=1, outer_min=8, outer_max=8, lag=lag, ring_slots=ring)
    m = _model(w.prog, w.trips, per_instr)
    assert m.barrier_loops == [w.prog.loop_id("O")]
    for s in range(8):
        out = explore(m, s, issue_bias=(0.3, 0.6, 0.9, 0.99)[s % 4])
        assert out.ok, (s, out)


def test_planted_missing_fallback_barrier_is_unsafe():
    """Without the barriers the consumer of a fallback dependency issues
    before its producer retired in some schedule."""
    w = lag_pipeline_workload(seed=2, n_wg=1, outer_min=8, outer_max=8)
    m = _model(w.prog, w.trips, False, barrier_loops=())
    kinds = set()
    for s in range(30):
        out = explore(m, s, issue_bias=0.95)
        if not out.ok:
            kinds.add(out.kind)
    assert kinds == {"unsafe"}


def test_lag_pipeline_plan():
    """Both ring dependencies of the lag-2 pipeline fall back; the store's
    dependency is C2 with one counter."""
    w = lag_pipeline_workload()
    p = Plan(w.prog, fallback=True)
    assert p.stats()["n_fallback"] == 2
    assert [f["kase"] for f in p.formulas()] == [KASE_FALLBACK, KASE_FALLBACK, 2]


def _fig_dep_nested(k, backward):
    """Fig. dep-nested: A{ B{ E0: x, prd, y }; E1: cns } (forward) or
    A{ E1: cns; B{ E0: x, prd, y } } (backward)."""
    from workloads.program import OP_NOP, ProgramBuilder
    b = ProgramBuilder("interp", n_engines=2)
    with b.loop("A"):
        if backward:
            b.instr(1, OP_NOP, name="cns")
        with b.loop("B"):
            b.instr(0, OP_NOP, name="x")
            b.instr(0, OP_NOP, name="prd")
            b.instr(0, OP_NOP, name="y")
        if not backward:
            b.instr(1, OP_NOP, name="cns")
    b.dep("prd", "cns", k)
    return b.build()


def test_cases_pinned_on_fig_dep_nested():
    """Section 5.2 on the nested example: forward admits offset 0 only,
    backward offset 1 only, backward offset 0 can never be met; every other
    offset falls back."""
    want = {(0, False): cases.C2, (1, False): cases.FALLBACK, (2, False): cases.FALLBACK,
            (0, True): cases.ORDER, (1, True): cases.C3, (2, True): cases.FALLBACK, (3, True): cases.FALLBACK}
    for (k, bwd), case in want.items():
        prog = _fig_dep_nested(k, bwd)
        got = cases.classify(prog, 0)
        assert got[0] == case and got[1] == prog.loop_id("A") and got[2] == prog.loop_id("B"), (k, bwd, got)
        assert got[3] == (not bwd)


def test_cases_pinned_on_eq1_brute_force():
    """The cases agree with the Eq. 1 counts the oracle brute-forces: C1 owes
    r_S - k once rhat_S > k, C2 owes r_P, C3 owes r_P once rhat_S > 1, at
    every consumer instance; fallback dependencies break the r_P form at some
    instance in some program (so no single register suffices)."""
    broken = 0
    for seed, prog, tt in _nests(400):
        trips, off = tt.flat()
        res = core.run(prog, trips, off[0], 0)
        for d in range(len(prog.deps)):
            case, S, P, _ = cases.classify(prog, d)
            k = prog.deps[d][2]
            r = res.recs[res.recs["dep"] == d]
            cnt, rP, hS = r["count_thr"].astype(int), r["r_P"].astype(int), r["rhat_S"].astype(int)
            if case == cases.C1:
                assert np.array_equal(cnt, np.where(hS > k, rP - k, 0)), (seed, d)
            elif case == cases.C2:
                assert np.array_equal(cnt, rP), (seed, d)
            elif case == cases.C3:
                assert np.array_equal(cnt, np.where(hS > 1, rP, 0)), (seed, d)
            elif case == cases.FALLBACK:
                fits = any(np.array_equal(cnt, np.where(hS > k, rP - j, 0)) for j in range(0, k + 2))
                broken += not fits
    assert broken >= 8
