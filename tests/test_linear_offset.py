"""The linearized-offset dependency (an EXTENSION, not in the paper): the
offset counts iterations of the shared loop across its trips.  Checked on
the CPU: a worked example against its closed form, the planner's thresholds
against the oracle's brute force over random nests, the classification, and
race coverage of a ring indexed across trips."""
import copy

import numpy as np
import pytest

from oracle import cases, core, hazard
from paper_2608_13757_amd import BfsError, Plan, bfs
from workloads import TripTables, random_nest, ring_workload
from workloads.program import OP_NOP, ProgramBuilder


def _nested_example(k, linear):
    """A{ B{ E0: prd; E1: cns } } (Fig. dep-general's nest)."""
    b = ProgramBuilder("interp", n_engines=2)
    with b.loop("A"):
        with b.loop("B"):
            b.instr(0, OP_NOP, name="prd")
            b.instr(1, OP_NOP, name="cns")
    b.dep("cns", "prd", k, linear=linear)
    return b.build()


def test_worked_example_closed_form():
    """B runs 3 then 4 times: with the linearized offset k = 2 the producer
    instance owed to the j-th consumer (j counted over both trips) is j - 2,
    also at the start of the second trip, where the paper's relation owes
    nothing (its counts are 0, 0, 1, 0, 0, 4, 5)."""
    prog = _nested_example(2, True)
    tt = TripTables([[np.array([1], np.int32), np.array([2], np.int32), np.array([3, 4], np.int32)]])
    trips, off = tt.flat()
    res = core.run(prog, trips, off[0], 0)
    lin = core.linearized_records(prog, res, 0)
    assert list(lin["count_thr"]) == [max(j - 2, 0) for j in range(1, 8)]
    assert list(res.recs["count_thr"]) == [0, 0, 1, 0, 0, 4, 5]
    plan = Plan(prog)
    f = plan.formulas()[0]
    assert (f["kase"], f["needs_mask"], f["expr_sub"]) == (cases.LINEAR, 0, 2)
    got = [plan.eval_threshold(0, int(r["r_P"]), int(r["rhat_S"])) for r in res.recs]
    assert got == list(lin["sem_thr"])


def test_planner_thresholds_match_brute_force():
    """Random nests with every allocatable producer-in-S dependency read
    linearized: the library's threshold equals the brute force at every
    consumer instance (per-loop counters, any N and K)."""
    checked = 0
    rng = np.random.default_rng(5)
    for seed in range(400):
        prog, tt = random_nest(seed, max_trip=4 if seed % 2 else 3)
        keep, lin = [], []
        for d, dep in enumerate(prog.deps):
            case, S, P, fwd = cases.classify(prog, d)
            if case == cases.C1:
                keep.append(dep)
                lin.append(int(rng.random() < 0.7))
        if not keep:
            continue
        prog = copy.deepcopy(prog)
        prog.deps, prog.dep_linear = keep, lin
        try:
            plan = Plan(prog)
        except BfsError:
            continue            # more counters than slots, or another resource limit
        trips, off = tt.flat()
        res = core.run(prog, trips, off[0], 0)
        for d in range(len(prog.deps)):
            recs = res.recs[res.recs["dep"] == d]
            want = core.linearized_records(prog, res, d)["sem_thr"] if lin[d] else recs["sem_thr"]
            got = [plan.eval_threshold(d, int(r["r_P"]), int(r["rhat_S"])) for r in recs]
            assert got == [int(x) for x in want], (seed, d)
            checked += len(recs)
    assert checked > 1500


def test_linear_needs_producer_in_s():
    b = ProgramBuilder("interp", n_engines=2)
    with b.loop("A"):
        b.instr(1, OP_NOP, name="cns")
        with b.loop("B"):
            b.instr(0, OP_NOP, name="prd")
    b.dep("prd", "cns", 1, linear=True)
    prog = b.build()
    assert cases.classify(prog, 0)[0] == cases.NOT_ALLOCATABLE
    with pytest.raises(BfsError) as e:
        Plan(prog)
    assert e.value.status == bfs.E_NOT_ALLOCATABLE


def test_ring_across_trips_race_coverage():
    """The ring indexed by the monotone register of B: covered by the
    linearized CONS->LOAD alone; the same dependency read with the paper's
    relation leaves the reuses that straddle a trip boundary unordered; the
    paper's ACQ form is covered."""
    w = ring_workload(seed=1, linear=True)
    trips, off = w.trips.flat()
    res = core.run(w.prog, trips, off[0], 0, w.base, w.x, 256)
    thr = res.recs["sem_thr"].copy()
    idx = np.nonzero(res.recs["dep"] == 1)[0]
    thr[idx] = core.linearized_records(w.prog, res, 1)["sem_thr"]
    assert hazard.check(w.prog, res, thresholds=thr) == []
    assert hazard.check(w.prog, res) != []
    w2 = ring_workload(seed=1, linear=False)
    res2 = core.run(w2.prog, trips, off[0], 0, w2.base, w2.x, 256)
    assert hazard.check(w2.prog, res2) == []
    # both forms compute the same values
    assert np.array_equal(res.out, res2.out)
