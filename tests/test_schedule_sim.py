"""Bisimulation by testing (Appendix A.2-A.5): random schedules of the
specification and implementation transition systems agree at every
reachable state, run to completion and end in the sequential datapath state;
planted mistakes in the implementation's thresholds or semaphore updates are
caught."""
import copy

import pytest

from paper_2608_13757_amd import ALLOC_PER_INSTR, ALLOC_PER_LOOP, BfsError, Plan
from tests.schedule_sim import Model, _listing, _parents, explore
from workloads import chain_workload, random_nest, stream_workload


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


def _model(prog, tt, per_instr, **kw):
    plan = Plan(prog, alloc=ALLOC_PER_INSTR if per_instr else ALLOC_PER_LOOP)
    trips, off = tt.flat()
    return Model(prog, plan, trips, off[0], per_instr=per_instr, **kw)


def test_random_nests_both_systems_agree():
    """Every reachable state of 4 random schedules per nest and allocation:
    the semaphore check admits exactly the instances whose Eq. 1 predicate
    holds, no schedule deadlocks."""
    programs = states = 0
    for seed in range(120):
        prog, tt = random_nest(seed, max_trip=4 if seed % 2 else 3)
        prog.deps = _allocatable(prog)
        if not prog.deps:
            continue
        for per_instr in (False, True):
            m = _model(prog, tt, per_instr)
            for s in range(4):
                out = explore(m, 1000 * seed + s, issue_bias=(0.2, 0.5, 0.8, 0.95)[s])
                assert out.ok, (seed, per_instr, s, out)
                states += out.steps
            programs += 1
    assert programs > 150 and states > 20000


@pytest.mark.parametrize("per_instr", [False, True])
def test_chain_schedules_values(per_instr):
    """The two-engine chain: random schedules end in the sequential state
    (the ring slot reuse and the accumulator are ordered by the plan)."""
    w = chain_workload(seed=1)
    m = _model(w.prog, w.trips, per_instr)
    for s in range(20):
        out = explore(m, s, issue_bias=0.3 + 0.03 * s)
        assert out.ok, (s, out)


@pytest.mark.parametrize("layout,inner_war", [("inplace", False), ("inplace", True), ("two_rings", True)])
@pytest.mark.parametrize("per_instr", [False, True])
def test_stream_schedules_values(layout, inner_war, per_instr):
    """The three-engine stream program on one workgroup of 3 O iterations."""
    w = stream_workload(seed=2, n_wg=1, outer=3, with_data=False, layout=layout, inner_war=inner_war,
                        n_gen=32 if layout == "inplace" else 8)
    m = _model(w.prog, w.trips, per_instr)
    for s in range(6):
        out = explore(m, s, issue_bias=(0.3, 0.6, 0.9)[s % 3])
        assert out.ok, (s, out)


def test_per_loop_counter_decode_matches_listing():
    """N is the number of the producer engine's instructions in the producer's
    loop body, K the producer's 1-based position among them."""
    for seed in range(120):
        prog, _ = random_nest(seed)
        prog.deps = _allocatable(prog)
        if not prog.deps:
            continue
        par, order = _parents(prog), _listing(prog)
        for f in Plan(prog).formulas():
            prd = prog.deps[f["dep"]][0]
            group = [i for i in order[par[prd]] if prog.instrs[i].engine == prog.instrs[prd].engine]
            assert f["loop_P"] == par[prd]
            assert f["N"] == len(group) and f["K"] == group.index(prd) + 1, (seed, f)


def _caught(prog, tt, kinds, per_instr=False, **kw):
    m = _model(prog, tt, per_instr, **kw)
    for s in range(40):
        out = explore(m, s, issue_bias=(0.2, 0.5, 0.9)[s % 3])
        if not out.ok:
            assert out.kind in kinds, out
            return True
    return False


def test_planted_threshold_one_short_is_unsafe():
    w = chain_workload(seed=1)
    for d in range(len(w.prog.deps)):
        assert _caught(w.prog, w.trips, {"unsafe"}, threshold_delta={d: -1}), d


def test_planted_threshold_one_over_blocks():
    w = chain_workload(seed=1)
    for d in range(len(w.prog.deps)):
        assert _caught(w.prog, w.trips, {"blocked"}, threshold_delta={d: 1}), d


def test_planted_missing_update_blocks():
    """A producer that never increments its semaphore: the consumer waits
    with its dependency met."""
    w = stream_workload(seed=2, n_wg=1, outer=2, with_data=False)
    plan = Plan(w.prog)
    f = plan.formulas()[0]
    prd = w.prog.deps[f["dep"]][0]
    assert _caught(w.prog, w.trips, {"blocked"}, drop_updates=[(prd, f["counter"])])


def test_planted_dropped_dependency_races():
    """Without the in-place ring's O-level acquire the values differ from the
    sequential ones in some schedule (the race the hazard check reports)."""
    w = stream_workload(seed=2, n_wg=1, outer=4, with_data=False)
    prog = copy.deepcopy(w.prog)
    prog.deps = [d for d in prog.deps if prog.instrs[d[1]].name != "ACQ_O"]
    assert _caught(prog, w.trips, {"values"})


@pytest.mark.parametrize("per_instr", [False, True])
def test_rmsnorm_adamw_schedules(per_instr):
    """The paper's software-pipelined RMSNorm and AdamW programs (offsets
    {0, 2}) on one workgroup of 7 steps: both issue predicates agree at every
    reachable state and no schedule deadlocks."""
    from workloads import adamw_program, adamw_worklist, rmsnorm_program, rmsnorm_worklist
    cases = [(rmsnorm_program(7, 1024, 2), rmsnorm_worklist(7, 1)[1]),
             (rmsnorm_program(7, 1024, 1, 1, 3), rmsnorm_worklist(7, 1)[1]),
             (adamw_program(7 * 256, 256, 2, 2), adamw_worklist(7 * 256, 256, 1)[1])]
    for prog, tt in cases:
        m = _model(prog, tt, per_instr)
        for s in range(6):
            out = explore(m, s, issue_bias=(0.3, 0.6, 0.95)[s % 3])
            assert out.ok, (s, out)
