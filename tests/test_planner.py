"""Planner (bfs_plan_create and friends) against the CPU oracle; no GPU needed.

Thresholds must equal the oracle's brute force of Eq. (1) bit-exactly, for
every consumer instance, in both counter units (per-loop semaphore values,
Section 5.5) and completion counts (per-instruction semaphores, Section 5.4),
and the barrier-mode static ordinals (Section 3.4)."""
import copy
import os
import re

import numpy as np
import pytest

from oracle import core
from paper_2608_13757_amd import (ALLOC_PER_ENGINE, ALLOC_PER_INSTR, ALLOC_PER_LOOP, MODE_BARRIER,
                                  MODE_BARRIER_FREE, BfsError, Plan, bfs)
from tests import fixtures
from workloads import (OP_NOP, ProgramBuilder, TripTables, attn_program, attn_worklist, chain_workload,
                       draw_trips, gemm_program, gemm_trips, random_nest, stream_program, stream_workload)

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _accepted_deps(prog):
    """Split deps into accepted / rejected by planning each one alone."""
    ok, rejected = [], []
    for d in prog.deps:
        q = copy.deepcopy(prog)
        q.deps = [d]
        try:
            Plan(q)
            ok.append(d)
        except BfsError as e:
            rejected.append((d, e.status))
    return ok, rejected


def _paper_case(prog, d):
    """The allocatable cases of Section 5.2, restated: returns 'C1', 'C2',
    'C3', 'order' or 'not-allocatable' for dependency d."""
    p, c, k = d
    par = {}
    for l, items in enumerate(prog.body):
        for kind, bid in items:
            if kind == 0:
                for i in prog.blocks[bid]:
                    par[i] = l

    def path(l):
        out = []
        while l >= 0:
            out.append(l)
            l = prog.loop_parent[l]
        return out[::-1]
    pp, pc = path(par[p]), path(par[c])
    S = [a for a, b in zip(pp, pc) if a == b][-1]

    def pos(i):
        l = par[i]
        if l == S:
            for j, (kind, bid) in enumerate(prog.body[S]):
                if kind == 0 and i in prog.blocks[bid]:
                    return (j, prog.blocks[bid].index(i))
        child = l
        while prog.loop_parent[child] != S:
            child = prog.loop_parent[child]
        return (prog.body[S].index((1, child)), -1)
    fwd = pos(p) < pos(c)
    if par[p] == S:
        return "order" if (not fwd and k == 0) else "C1"
    if fwd:
        return "C2" if k == 0 else "not-allocatable"
    if k == 0:
        return "order"
    return "C3" if k == 1 else "not-allocatable"


def _check_against_oracle(prog, tt):
    trips, off = tt.flat()
    res = core.run(prog, trips, off[0], 0)
    pl = Plan(prog, MODE_BARRIER_FREE, ALLOC_PER_LOOP)
    pi = Plan(prog, MODE_BARRIER_FREE, ALLOC_PER_INSTR)
    pb = Plan(prog, MODE_BARRIER, ALLOC_PER_LOOP)
    for rec in res.recs:
        d, rP, rh = int(rec["dep"]), int(rec["r_P"]), int(rec["rhat_S"])
        assert pl.eval_threshold(d, rP, rh) == rec["sem_thr"], (d, rec)
        assert pi.eval_threshold(d, rP, rh) == rec["count_thr"], (d, rec)
        assert pb.eval_threshold(d, rP, rh) == rec["barrier_thr"], (d, rec)
        assert rec["order_ok"]
    return len(res.recs)


def _check_linear_against_oracle(prog, tt):
    """Like _check_against_oracle for a program with linearized
    dependencies: those are checked against the brute force of the
    linearized relation (both allocations), the others against Eq. 1's
    records (both allocations and the barrier mode)."""
    trips, off = tt.flat()
    res = core.run(prog, trips, off[0], 0)
    pl = Plan(prog, MODE_BARRIER_FREE, ALLOC_PER_LOOP)
    pi = Plan(prog, MODE_BARRIER_FREE, ALLOC_PER_INSTR)
    pb = Plan(prog, MODE_BARRIER, ALLOC_PER_LOOP)
    n = 0
    for d in range(len(prog.deps)):
        recs = res.recs[res.recs["dep"] == d]
        lin = bool(prog.dep_linear and prog.dep_linear[d])
        want = core.linearized_records(prog, res, d) if lin else recs
        for rec, w in zip(recs, want):
            rP, rh = int(rec["r_P"]), int(rec["rhat_S"])
            assert pl.eval_threshold(d, rP, rh) == w["sem_thr"], (d, rec)
            assert pi.eval_threshold(d, rP, rh) == w["count_thr"], (d, rec)
            if not lin:
                assert pb.eval_threshold(d, rP, rh) == rec["barrier_thr"], (d, rec)
                assert rec["order_ok"]
        n += len(recs)
    return n


def test_random_nests_bit_exact():
    n_checked, cases = 0, set()
    for seed in range(1200):
        prog, tt = random_nest(seed, max_trip=4 if seed % 2 else 3)
        ok, rejected = _accepted_deps(prog)
        for d, st in rejected:
            want = _paper_case(prog, d)
            assert want in ("order", "not-allocatable"), (seed, d, want)
            assert st == (bfs.E_ORDER if want == "order" else bfs.E_NOT_ALLOCATABLE)
        for d in ok:
            cases.add(_paper_case(prog, d))
        if not ok:
            continue
        prog.deps = ok
        n_checked += _check_against_oracle(prog, tt)
    assert n_checked > 5000
    assert cases == {"C1", "C2", "C3"}


@pytest.mark.parametrize("name", fixtures.all_fixtures())
def test_paper_figures_through_planner(name):
    fx, prog, tt = fixtures.load(name)
    _check_against_oracle(prog, tt)


def test_per_scope_figure_formula():
    """Fig. per-scope-example-alloc: w = isGT(rhat_A, 0) * (2 * r_A)."""
    fx, prog, tt = fixtures.load("fig_per_scope.json")
    f = Plan(prog).formulas()[0]
    assert (f["kase"], f["N"], f["K"], f["k"], f["needs_mask"]) == (1, 2, 2, 0, 0)
    p = Plan(prog)
    assert [p.eval_threshold(0, a, a) for a in (1, 2, 3)] == [2, 4, 6]
    fi = Plan(prog, alloc=ALLOC_PER_INSTR)
    assert [fi.eval_threshold(0, a, a) for a in (1, 2, 3)] == [1, 2, 3]


def test_dep_nested_cases():
    fx, prog, tt = fixtures.load("fig_dep_nested.json")
    f = Plan(prog).formulas()
    assert f[0]["kase"] == 2 and f[1]["kase"] == 3
    assert f[0]["loop_P"] == f[1]["loop_P"] == prog.loop_id("B")


def test_workload_programs():
    for prog, tt in [(chain_workload(0).prog, chain_workload(0).trips)]:
        _check_against_oracle(prog, tt)
    s = stream_workload(seed=0, n_wg=1, outer=5, with_data=False)
    _check_against_oracle(s.prog, s.trips)
    g = gemm_program(512, 256, 128)
    _check_against_oracle(g, TripTables([gemm_trips(512, 256, 128).per_wg[0]]))
    for lengths in ([1], [64], [65], [300], [300, 65, 1, 129]):
        # one workgroup runs every tile: the T loop spans several tiles
        _check_linear_against_oracle(attn_program(2), attn_worklist(lengths, 2, n_wg=1).trips)
    # the second workloads of the paper's suite and the MoE program
    from workloads import adamw_program, adamw_worklist, moe_program, moe_worklist, rmsnorm_program, \
        rmsnorm_worklist
    for rows in (1, 2, 7):
        _, tt = rmsnorm_worklist(rows, 1)
        _check_against_oracle(rmsnorm_program(rows, 1024, 2), tt)
        _check_against_oracle(rmsnorm_program(rows, 1024, 2, 1, 3), tt)
    for n in (256, 3000, 8192):
        _, tt = adamw_worklist(n, 1024, 1)
        _check_against_oracle(adamw_program(n, 1024, 2, 2), tt)
        _check_against_oracle(adamw_program(n, 1024, 2, 3), tt)
    for ph in (1, 2):
        wl = moe_worklist(np.array([300, 0, 129, 1, 530]), ph, 256, 256)
        for w in range(0, len(wl.trips.per_wg), 3):
            _check_against_oracle(moe_program(ph, 256, 256), TripTables([wl.trips.per_wg[w]]))


def test_moe_linear_ring_thresholds():
    """The MoE program with MMA->LOAD read linearized (an extension): the
    planner's thresholds equal the brute force of the linearized relation at
    every consumer instance, across M-tile boundaries (runs of 2 and 3
    M-tiles), and the paper's relation for every other dependency."""
    from workloads import moe_program, moe_worklist
    checked = 0
    for ph in (1, 2):
        prog = moe_program(ph, 256, 256, ring=3, linear=True)
        d_lin = [i for i, (p, c, k) in enumerate(prog.deps)
                 if (prog.instrs[p].name, prog.instrs[c].name) == ("MMA", "LOAD")]
        assert d_lin and prog.dep_linear[d_lin[0]] == 1
        assert not any((prog.instrs[p].name, prog.instrs[c].name) == ("MMA", "ACQL") for p, c, k in prog.deps)
        plan = Plan(prog)
        assert plan.formulas()[d_lin[0]]["kase"] == 6
        wl = moe_worklist(np.array([300, 0, 129, 1, 530]), ph, 256, 256, mchunk=3)
        for per in wl.trips.per_wg:
            if int(per[1][0]) < 2:
                continue
            tt = TripTables([per])
            trips, off = tt.flat()
            res = core.run(prog, trips, off[0], 0)
            for d in range(len(prog.deps)):
                recs = res.recs[res.recs["dep"] == d]
                want = core.linearized_records(prog, res, d)["sem_thr"] if d == d_lin[0] else recs["sem_thr"]
                got = [plan.eval_threshold(d, int(r["r_P"]), int(r["rhat_S"])) for r in recs]
                assert got == [int(x) for x in want], (ph, d)
                checked += len(recs)
    assert checked > 200


def test_moe_worklist_covers_every_tile_once():
    """Every (expert, output tile, M-tile) of both phases appears in exactly
    one work item, runs hold at most the default run length of M-tiles,
    trips match; both M-tile heights."""
    from workloads import MOE_BN, moe_worklist
    from workloads.configs import MOE_MCHUNKS, moe_chunks
    from workloads.tensors import zipf_counts
    for bm in (128, 256):
        for counts in (zipf_counts(32768, 64), np.array([300, 0, 129, 1, 530])):
            for ph, (hidden, ffn) in ((1, (4096, 1408)), (2, (4096, 1408)), (1, (256, 256)), (2, (256, 256))):
                wl = moe_worklist(counts, ph, hidden, ffn, bm=bm)
                n_dim = ffn if ph == 1 else hidden
                seen = set()
                for (e, n0, mt0, n_mt), tr in zip(wl.work.tolist(), wl.trips.per_wg):
                    assert int(tr[1][0]) == n_mt and len(tr[2]) == n_mt and n_mt <= MOE_MCHUNKS[bm]
                    assert all(int(c) == moe_chunks(ph, bm) for c in tr[3])
                    for m in range(mt0, mt0 + n_mt):
                        key = (e, n0, m)
                        assert key not in seen
                        seen.add(key)
                want = {(e, n0, m) for e in range(len(counts)) for n0 in range(0, n_dim, MOE_BN[ph])
                        for m in range(-(-int(counts[e]) // bm))}
                assert seen == want


def test_fused_family_formulas():
    """The dependencies of the GEMM and attention programs land in the cases
    the kernels rely on: ring reuse as C1 backward with the ring depth, the
    epilogue-after-K-loop and final-row-sum dependencies as C2."""
    g = gemm_program(512, 256, 128)
    fg = {(g.instrs[p].name, g.instrs[c].name): f for (p, c, k), f in zip(g.deps, Plan(g).formulas())}
    assert fg[("MMA", "LOAD")]["kase"] == 1 and fg[("MMA", "LOAD")]["k"] == 4 and not fg[("MMA", "LOAD")]["forward"]
    assert fg[("MMA", "SPILL")]["kase"] == 2 and fg[("BIAS", "SPILL")]["kase"] == 1
    for linear in (True, False):
        a = attn_program(16, nk=3, nv=2, linear=linear)
        fa = {(a.instrs[p].name, a.instrs[c].name): f for (p, c, k), f in zip(a.deps, Plan(a).formulas())}
        assert fa[("QK", "LOADK")]["k"] == 3 and fa[("PV", "LOADV")]["k"] == 2 and fa[("PREAD", "QK")]["k"] == 2
        assert all(fa[x]["kase"] == 1 for x in [("LOADK", "QK"), ("QK", "SM"), ("SM", "PREAD"), ("LOADV", "PV")])
        reuse = [("QK", "LOADK"), ("PV", "LOADV"), ("PREAD", "QK")]
        assert all(fa[x]["kase"] == (6 if linear else 1) for x in reuse)
        if not linear:
            # the acquires drain the previous tile: C3 at T, offset 1
            for x in [("QK", "ACQK"), ("PV", "ACQV"), ("PREAD", "ACQS")]:
                assert fa[x]["kase"] == 3 and fa[x]["k"] == 1 and fa[x]["loop_S"] == a.loop_id("T")
        assert fa[("SM", "NORM")]["kase"] == 2
        assert fa[("NORM", "SM")]["kase"] == 1 and fa[("NORM", "SM")]["loop_S"] == a.loop_id("T")
    # the work list covers every (sequence, head, query tile) once; tile j of
    # workgroup w sits at row w + j * n_wg, on w's XCD (w % 8) with every
    # tile of its (sequence, head)
    for n_wg in (1, 5, 16, 256):
        wl = attn_worklist([1, 64, 129, 300, 4096], 3, n_wg=n_wg)
        seen, xcd_of_pair = [], {}
        for w, per in enumerate(wl.trips.per_wg):
            n_t = int(per[1][0])
            assert len(per[2]) == n_t
            for j in range(n_t):
                r = wl.work[w + j * n_wg]
                assert r[1] > 0 and int(per[2][j]) == -(-int(r[1]) // 64)
                seen.append(tuple(r))
                if n_wg >= 8:
                    assert xcd_of_pair.setdefault((int(r[0]), int(r[3])), w % 8) == w % 8
        assert len(seen) == len(set(seen)) == 3 * (1 + 1 + 2 + 3 + 32)


def test_rejections():
    b = ProgramBuilder("interp", 2)
    with b.loop("A"):
        b.instr(1, OP_NOP, name="c")
        b.instr(0, OP_NOP, name="p")
    b.dep("p", "c", 0)                       # same-region backward at offset 0
    with pytest.raises(BfsError) as e:
        Plan(b.build())
    assert e.value.status == bfs.E_ORDER

    b = ProgramBuilder("interp", 2)
    with b.loop("A"):
        with b.loop("B"):
            b.instr(0, OP_NOP, name="p")
        b.instr(1, OP_NOP, name="c")
    b.dep("p", "c", 1)                       # nested forward with offset 1
    with pytest.raises(BfsError) as e:
        Plan(b.build())
    assert e.value.status == bfs.E_NOT_ALLOCATABLE

    b = ProgramBuilder("interp", 2)
    with b.loop("A"):
        b.instr(1, OP_NOP, name="c")
        with b.loop("B"):
            b.instr(0, OP_NOP, name="p")
    b.dep("p", "c", 2)                       # nested backward with offset 2
    with pytest.raises(BfsError) as e:
        Plan(b.build())
    assert e.value.status == bfs.E_NOT_ALLOCATABLE


def test_malformed_programs():
    w = chain_workload(0)
    base = w.prog.flat()
    bad = dict(base)
    bad["instr_engine"] = [0, 5, 1, 1]       # engine out of range
    with pytest.raises(BfsError) as e:
        Plan(bad)
    assert e.value.status == bfs.E_INVALID
    bad = dict(base)
    bad["deps"] = [(0, 0, 0)]                # self dependency
    with pytest.raises(BfsError):
        Plan(bad)
    bad = dict(base)
    bad["loop_parent"] = [-1, 0, 0]          # loop listed outside its parent
    with pytest.raises(BfsError):
        Plan(bad)


def test_resource_stats():
    s = stream_workload(seed=0, n_wg=1, outer=2, with_data=False)
    pl, pi, pb = Plan(s.prog), Plan(s.prog, alloc=ALLOC_PER_INSTR), Plan(s.prog, MODE_BARRIER)
    st_l, st_i, st_b = pl.stats(), pi.stats(), pb.stats()
    assert st_l["salu_ops_per_wait"] == 5 and st_i["salu_ops_per_wait"] == 3
    assert st_b["n_counters"] == 3 and st_b["regs_per_engine"] == 0
    assert st_l["n_waits"] == len(s.prog.deps)
    # one counter per (loop, engine) pair that some dependency reads
    pairs = {(f["loop_P"], f["prd_engine"]) for f in pl.formulas()}
    assert st_l["n_counters"] == len(pairs)


def test_per_engine_plans():
    """Per-engine allocation (Section 6.1): one counter per producer engine
    that every instruction of the engine increments; each dependency keeps
    k + 1 snapshots when its producer sits directly in S, else one; host
    evaluation is refused (the thresholds are snapshots of the walk)."""
    s = stream_workload(seed=0, n_wg=1, outer=2, with_data=False, layout="two_rings", n_gen=8, inner_war=True)
    pe, pl = Plan(s.prog, alloc=ALLOC_PER_ENGINE), Plan(s.prog)
    fe, fl = pe.formulas(), pl.formulas()
    prd_engines = {f["prd_engine"] for f in fe}
    assert pe.stats()["n_counters"] == len(prd_engines) < pl.stats()["n_counters"]
    for f, g in zip(fe, fl):
        assert (f["kase"], f["loop_S"], f["loop_P"], f["k"]) == (g["kase"], g["loop_S"], g["loop_P"], g["k"])
        assert f["snap_slots"] == (f["k"] + 1 if f["loop_P"] == f["loop_S"] else 1)
        assert g["snap_slots"] == 0
    slot = {f["prd_engine"]: f["counter"] for f in fe}
    assert len(set(slot.values())) == len(slot)
    assert pe.stats()["salu_ops_per_wait"] == 3
    assert pe.stats()["regs_per_engine"] > pl.stats()["regs_per_engine"]
    with pytest.raises(BfsError) as e:
        pe.eval_threshold(0, 1, 1)
    assert e.value.status == bfs.E_UNSUPPORTED
    # barrier mode ignores the allocation
    assert Plan(s.prog, MODE_BARRIER, ALLOC_PER_ENGINE).static_waits() == Plan(s.prog, MODE_BARRIER).static_waits()


def test_abi_exports_every_header_symbol():
    hdr = open(os.path.join(ROOT, "include", "bfs.h")).read()
    names = set(re.findall(r"^\s*(?:const\s+)?[a-z_]+\s*\*?\s*(bfs_[a-z_]+)\s*\(", hdr, re.M))
    assert names == set(bfs.EXPORTED), names ^ set(bfs.EXPORTED)
    L = bfs.lib()
    for n in names:
        assert hasattr(L, n), n


def _mutate(f, rng):
    """A copy of flat program ``f`` with random contents: every array keeps
    the length its counts and offsets imply (the caller's side of the C
    ABI's contract), every entry may be out of range."""
    g = copy.deepcopy(f)
    n_loops, n_instrs = len(g["loop_parent"]), len(g["instr_engine"])
    n_body, n_blk = len(g["body_kind"]), len(g["block_off"]) - 1
    bad = lambda lo, hi: int(rng.integers(lo, hi + 1))
    for _ in range(int(rng.integers(1, 5))):
        what = int(rng.integers(0, 14))
        if what == 0 and n_loops:
            g["loop_parent"][bad(0, n_loops - 1)] = bad(-3, n_loops + 2)
        elif what == 1 and n_loops:
            g["loop_is_cond"][bad(0, n_loops - 1)] = bad(-1, 3)
        elif what == 2 and n_loops > 1:
            g["body_off"][bad(1, n_loops - 1)] = bad(-2, n_body + 2)
        elif what == 3 and n_body:
            g["body_kind"][bad(0, n_body - 1)] = bad(-2, 3)
        elif what == 4 and n_body:
            g["body_id"][bad(0, n_body - 1)] = bad(-3, max(n_loops, n_blk) + 3)
        elif what == 5 and n_blk > 1:
            g["block_off"][bad(1, n_blk - 1)] = bad(-2, len(g["block_instrs"]) + 2)
        elif what == 6 and g["block_instrs"]:
            g["block_instrs"][bad(0, len(g["block_instrs"]) - 1)] = bad(-3, n_instrs + 3)
        elif what == 7 and n_instrs:
            g["instr_engine"][bad(0, n_instrs - 1)] = bad(-2, 10)
        elif what == 8 and n_instrs:
            g["instr_opcode"][bad(0, n_instrs - 1)] = bad(-2, 64)
        elif what == 9 and n_instrs:
            g["instr_args"][bad(0, n_instrs - 1)][bad(0, 7)] = bad(-5, 300)
        elif what == 10 and g["deps"]:
            d = list(g["deps"][bad(0, len(g["deps"]) - 1)])
            d[bad(0, 2)] = bad(-3, n_instrs + 3) if rng.random() < 0.7 else bad(-5, 40)
            g["deps"][bad(0, len(g["deps"]) - 1)] = tuple(d)
        elif what == 11:
            g["n_engines"] = bad(-1, 10)
        elif what == 12:
            g["waves_per_engine"][bad(0, 7)] = bad(-2, 12)
        elif what == 13:
            g["dep_linear"] = [bad(-1, 2) for _ in g["deps"]]
    return g


def test_planner_rejects_malformed_programs():
    """Random malformed programs through the C ABI: every call returns OK or
    an error status (never crashes), and every accepted plan answers its
    query calls.  Run under a sanitizer build of the planner, this also
    checks memory safety of the validation."""
    rng = np.random.default_rng(2024)
    bases = [random_nest(seed=s)[0].flat() for s in range(40)]
    bases += [gemm_program(512, 512, 256).flat(), attn_program(2).flat(), stream_program().flat()]
    valid = {getattr(bfs, n) for n in dir(bfs) if n.startswith("E_")} | {0}
    accepted = rejected = 0
    for i in range(600):
        g = _mutate(bases[i % len(bases)], rng)
        mode = int(rng.choice([MODE_BARRIER_FREE, MODE_BARRIER, 5]))
        alloc = int(rng.choice([ALLOC_PER_LOOP, ALLOC_PER_INSTR, ALLOC_PER_ENGINE, 7]))
        try:
            plan = Plan(g, mode, alloc)
        except BfsError as e:
            assert e.status in valid and e.status != 0
            rejected += 1
            continue
        accepted += 1
        plan.formulas()
        plan.stats()
        if mode == MODE_BARRIER:
            plan.static_waits()
        for d in range(len(g["deps"]) + 2):
            try:
                plan.eval_threshold(d, int(rng.integers(0, 9)), int(rng.integers(0, 9)))
            except BfsError as e:
                assert e.status in valid and e.status != 0
    assert rejected > 100 and accepted > 10
