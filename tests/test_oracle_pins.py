"""Pins of the CPU oracle against what the paper and the mathematics fix.

Nothing here compares the oracle with itself: expected values come from the
paper's worked figures (tests/golden, each with its citation), closed forms,
invariants that follow from the definitions, and plain library identities.
"""
import copy

import numpy as np
import pytest

from oracle import core, hazard, mathref
from tests import fixtures
from workloads import (OP_NOP, ProgramBuilder, TripTables, chain_workload,
                       draw_trips, random_nest, stream_workload)
from workloads.tensors import (attn_inputs, bf16_to_f32, gemm_inputs,
                               moe_inputs, to_bf16_bits, zipf_counts)


def _run(prog, tt, wg=0):
    trips, off = tt.flat()
    return core.run(prog, trips, off[wg], wg)


# --------------------------------------------------------------------------
# worked examples printed in the paper
# --------------------------------------------------------------------------
@pytest.mark.parametrize("name", fixtures.all_fixtures())
def test_paper_figure(name):
    fx, prog, tt = fixtures.load(name)
    res = _run(prog, tt)
    for dep, exp in fx["expected"].items():
        r = res.recs[res.recs["dep"] == int(dep)]
        if "count" in exp:
            assert r["count_thr"].tolist() == exp["count"], fx["citation"]
        if "sem" in exp:
            assert r["sem_thr"].tolist() == exp["sem"], fx["citation"]
        if "barrier" in exp:
            assert r["barrier_thr"].tolist() == exp["barrier"], fx["citation"]
        assert r["order_ok"].all()


def test_fixture_count():
    assert len(fixtures.all_fixtures()) >= 7


# --------------------------------------------------------------------------
# closed forms that follow directly from the definitions
# --------------------------------------------------------------------------
def _single_loop(n_prd_engine_instrs, k, trips, producer_pos):
    """loop A{ E0: n instructions; E1: cns } with dep (E0's instr at producer_pos, cns, k)."""
    b = ProgramBuilder("interp", 2)
    with b.loop("A"):
        for i in range(n_prd_engine_instrs):
            b.instr(0, OP_NOP, name=f"p{i}")
        b.instr(1, OP_NOP, name="cns")
    b.dep(f"p{producer_pos}", "cns", k)
    prog = b.build()
    tt = TripTables([draw_trips(prog, lambda l, n: np.asarray(trips[:n]))])
    return prog, tt


@pytest.mark.parametrize("n,kpos,k", [(1, 0, 0), (2, 1, 0), (3, 0, 0), (3, 2, 1), (4, 1, 3), (1, 0, 5)])
def test_single_loop_closed_form(n, kpos, k):
    """Producer and consumer in one loop executed once with trip 9: iteration
    i owes max(i - k, 0) producer completions (underflow when i <= k), and on
    a counter shared by the n instructions of engine 0, the c-th completion of
    the producer at 1-based position K leaves the counter at n*c - (n - K)."""
    prog, tt = _single_loop(n, k, [9], kpos)
    res = _run(prog, tt)
    i = np.arange(1, 10)
    count = np.maximum(i - k, 0)
    assert res.recs["count_thr"].tolist() == count.tolist()
    K = kpos + 1
    sem = np.where(count > 0, n * count - (n - K), 0)
    assert res.recs["sem_thr"].tolist() == sem.tolist()


def test_straight_line_ordinal():
    """Top-level straight line: threshold = producer's ordinal on its engine."""
    b = ProgramBuilder("interp", 3)
    names = []
    for i, e in enumerate([0, 1, 0, 2, 0, 1, 2, 0]):
        names.append(b.instr(e, OP_NOP, name=f"i{i}"))
    b.dep("i4", "i5", 0)     # i4 is engine 0's third instruction
    b.dep("i3", "i6", 0)     # i3 is engine 2's first instruction
    prog = b.build()
    res = _run(prog, TripTables([[np.array([1])]]))
    assert res.recs["sem_thr"].tolist() == [3, 1]
    assert res.recs["barrier_thr"].tolist() == [3, 1]


def test_final_counter_invariant():
    """Each per-loop counter ends at (its engine's instructions in that loop's
    body) x (total iterations of the loop) -- the trip table summed directly."""
    for seed in range(25):
        prog, tt = random_nest(seed)
        res = _run(prog, tt)
        per = np.zeros((prog.n_loops, prog.n_engines), np.int64)
        for l, items in enumerate(prog.body):
            for kind, bid in items:
                if kind == 0:
                    for i in prog.blocks[bid]:
                        per[l, prog.instrs[i].engine] += 1
        total = np.array([int(np.sum(t)) for t in tt.per_wg[0]])
        assert (res.final_cnt == per * total[:, None]).all()


def test_underflow_and_monotonicity():
    """No wait when the target's shared-loop component is <= 0 (Section 4.2),
    and owed counts never decrease within a trip of the shared loop."""
    for seed in range(25):
        prog, tt = random_nest(seed)
        res = _run(prog, tt)
        for d, (p, c, k) in enumerate(prog.deps):
            r = res.recs[res.recs["dep"] == d]
            under = r["rhat_S"] <= k
            assert (r["count_thr"][under] == 0).all()
            nz = r["count_thr"][r["count_thr"] > 0]
            assert (np.diff(nz) >= 0).all()


def test_zero_trip_loops_are_exercised():
    zero = 0
    for seed in range(25):
        prog, tt = random_nest(seed)
        zero += sum(int((t == 0).sum()) for t in tt.per_wg[0][1:])
    assert zero > 0


# --------------------------------------------------------------------------
# tile-machine values
# --------------------------------------------------------------------------
def test_chain_values_closed_form():
    """out = 0.5 * sum of every loaded tile (numpy sum, independent of the walk)."""
    w = chain_workload(seed=1)
    trips, off = w.trips.flat()
    out = core.values(w.prog, trips, off, w.base, w.x, 256)
    ref = 0.5 * w.x.astype(np.float64).sum(axis=0)
    assert np.abs(out - ref).max() < 1e-12
    assert w.n_tiles == int(np.sum(w.trips.per_wg[0][2]))


def test_stream_values_closed_form():
    s = stream_workload(seed=2, n_wg=3, outer=5)
    trips, off = s.trips.flat()
    out = core.values(s.prog, trips, off, s.base, s.x, s.n_tiles * 64)
    assert np.array_equal(out, s.x.astype(np.float64).reshape(-1) + 1.0)


# --------------------------------------------------------------------------
# hazard coverage (CPU race check) and planted mistakes
# --------------------------------------------------------------------------
@pytest.mark.parametrize("mode", ["barrier_free", "barrier"])
def test_hazard_coverage_of_workload_programs(mode):
    w = chain_workload(seed=0)
    trips, off = w.trips.flat()
    res = core.run(w.prog, trips, off[0], 0)
    assert hazard.check(w.prog, res, mode) == []
    s = stream_workload(seed=0, n_wg=2, outer=6, with_data=False)
    trips, off = s.trips.flat()
    res = core.run(s.prog, trips, off[1], 1)
    assert res.recs["order_ok"].all()
    assert hazard.check(s.prog, res, mode) == []


@pytest.mark.parametrize("layout", ["inplace", "two_rings"])
def test_stream_layouts_race_free(layout):
    """Both ring layouts of the stream program order every conflicting
    access (CPU happens-before check over whole workgroups)."""
    s = stream_workload(seed=4, n_wg=3, outer=12, with_data=False, layout=layout,
                        n_gen=32 if layout == "inplace" else 8)
    trips, off = s.trips.flat()
    for wg in range(3):
        res = core.run(s.prog, trips, off[wg], wg)
        assert hazard.check(s.prog, res, "barrier_free") == []
        assert hazard.check(s.prog, res, "barrier") == []


@pytest.mark.parametrize("layout", ["inplace", "two_rings"])
def test_stream_slot_reuse_within_a_trip_race_free(layout):
    """Two slots per generation with inner trips up to 4: the offset-per_gen
    dependencies order the reuse of a slot within one trip of I."""
    from workloads import stream_program
    s = stream_workload(seed=5, n_wg=2, outer=12, with_data=False, layout=layout, inner_war=True)
    p = stream_program(per_gen=2, inner_war=True, layout=layout)
    trips, off = s.trips.flat()
    assert int(trips.max()) >= 3
    for wg in range(2):
        res = core.run(p, trips, off[wg], wg)
        assert hazard.check(p, res, "barrier_free") == []
    bare = stream_program(per_gen=2, inner_war=False, layout=layout)
    assert hazard.check(bare, core.run(bare, trips, off[0], 0)) != []


def test_stream_inplace_needs_its_o_dependency_and_generations():
    """Planted mistakes the race check must catch: the in-place layout without
    MARK_O -> ACQ_O, and with too few generations for two O iterations."""
    s = stream_workload(seed=4, n_wg=2, outer=12, with_data=False)
    trips, off = s.trips.flat()
    p = copy.deepcopy(s.prog)
    p.deps = [d for d in p.deps if p.instrs[d[1]].name != "ACQ_O"]
    assert hazard.check(p, core.run(p, trips, off[0], 0)) != []
    from workloads import stream_program
    few = stream_program(n_gen=16)      # M trips up to 16: o and o + 2 may now share slots with o + 1
    assert hazard.check(few, core.run(few, trips, off[0], 0)) != []


def test_stream_inplace_trip_bounds():
    """The in-place ring (32 generations of 4 slots, MARK_O -> ACQ_O at
    offset 2, no inner reuse dependency) is race-free with every M trip at
    its bound n_gen / 2 = 16 and every I trip at per_gen = 4, and races
    one past either bound (the launcher reports such trips as invalid)."""
    from workloads import stream_fixed_trips, stream_program
    p = stream_program()
    ok = stream_fixed_trips(p, [16] * 6, 4)
    trips, off = ok.flat()
    res = core.run(p, trips, off[0], 0)
    assert res.recs["order_ok"].all()
    assert hazard.check(p, res, "barrier_free") == []
    for m_trips, i_trip in (([16, 17, 16, 16], 4), ([16] * 4, 5)):
        bad = stream_fixed_trips(p, m_trips, i_trip)
        trips, off = bad.flat()
        assert hazard.check(p, core.run(p, trips, off[0], 0), "barrier_free") != [], (m_trips, i_trip)
    # with the inner reuse dependency a trip of I may be longer than a generation
    pw = stream_program(inner_war=True)
    long_i = stream_fixed_trips(pw, [16] * 3, 9)
    trips, off = long_i.flat()
    assert hazard.check(pw, core.run(pw, trips, off[0], 0), "barrier_free") == []


def test_per_engine_counter_closed_forms():
    """The per-engine counter column (Section 6.1: one counter per engine,
    incremented by every instruction of the engine) against closed forms
    computed from the trip tables alone.

    Chain, engine 0 = {ACQ in A, LOAD in B}: right after the LOAD of B
    iteration r_B it has retired r_A ACQs and r_B LOADs, so LOAD -> CONS
    owes r_A + r_B.  Engine 1 = {CONS in B, STORE after A}: CONS -> LOAD
    (k = 4) owes [rhat_B > 4] (r_B - 4) and CONS -> ACQ (k = 1) owes
    [rhat_A > 1] r_B.  In-place stream, engine 2 = {STORE in I, MARK_O in O}:
    MARK_O -> ACQ_O (k = 2) at O iteration o owes the STOREs of O iterations
    1 .. o - 2 plus o - 2 markers; LOAD -> ADD owes r_O + r_I (one ACQ_O per
    O iteration, one LOAD per I iteration)."""
    w = chain_workload(seed=2)
    trips, off = w.trips.flat()
    res = core.run(w.prog, trips, off[0], 0)
    A, B = w.prog.loop_id("A"), w.prog.loop_id("B")
    names = {i: ins.name for i, ins in enumerate(w.prog.instrs)}
    cons_at = {}
    for d, (pp, cc, k) in enumerate(w.prog.deps):
        idx = np.nonzero(res.inst["instr"] == cc)[0]
        cons_at[(names[pp], names[cc])] = (d, idx)
    d, idx = cons_at[("LOAD", "CONS")]
    got = res.recs[res.recs["dep"] == d]["eng_thr"]
    assert np.array_equal(got, res.r_snap[idx, A] + res.r_snap[idx, B])
    d, idx = cons_at[("CONS", "LOAD")]
    got = res.recs[res.recs["dep"] == d]["eng_thr"]
    want = np.where(res.rhat_snap[idx, B] > 4, res.r_snap[idx, B] - 4, 0)
    assert np.array_equal(got, want) and want.max() > 0
    d, idx = cons_at[("CONS", "ACQ")]
    got = res.recs[res.recs["dep"] == d]["eng_thr"]
    want = np.where(res.rhat_snap[idx, A] > 1, res.r_snap[idx, B], 0)
    assert np.array_equal(got, want) and want.max() > 0

    s = stream_workload(seed=3, n_wg=2, outer=9, with_data=False)
    trips, off = s.trips.flat()
    res = core.run(s.prog, trips, off[1], 1)
    per = s.trips.per_wg[1]
    m_trips, i_trips = per[2], per[3]
    stores_upto = np.concatenate([[0], np.cumsum([int(i_trips[int(m_trips[:o].sum()):int(m_trips[:o + 1].sum())].sum())
                                                  for o in range(len(m_trips))])])
    names = {i: ins.name for i, ins in enumerate(s.prog.instrs)}
    O, I = s.prog.loop_id("O"), s.prog.loop_id("I")
    for d, (pp, cc, k) in enumerate(s.prog.deps):
        recs = res.recs[res.recs["dep"] == d]
        idx = np.nonzero(res.inst["instr"] == cc)[0]
        if (names[pp], names[cc]) == ("MARK_O", "ACQ_O"):
            o = res.r_snap[idx, O]
            want = np.where(o > 2, stores_upto[np.maximum(o - 2, 0)] + (o - 2), 0)
        elif (names[pp], names[cc]) == ("LOAD", "ADD"):
            want = res.r_snap[idx, O] + res.r_snap[idx, I]
        else:                                            # ADD -> STORE: engine 1 is the ADD alone
            want = res.r_snap[idx, I]
        assert np.array_equal(recs["eng_thr"], want), names[pp] + "->" + names[cc]


def test_per_engine_equals_per_loop_for_single_loop_engines():
    """Where every instruction of the producer's engine sits directly in the
    producer's loop, the per-engine and per-loop counters are the same
    counter (random nests)."""
    checked = 0
    for seed in range(120):
        prog, tt = random_nest(seed)
        trips, off = tt.flat()
        res = core.run(prog, trips, off[0], 0)
        parent = {}
        for l, items in enumerate(prog.body):
            for kind, bid in items:
                if kind == 0:
                    for i in prog.blocks[bid]:
                        parent[i] = l
        for d, (pp, cc, k) in enumerate(prog.deps):
            e = prog.instrs[pp].engine
            if all(parent[i] == parent[pp] for i, ins in enumerate(prog.instrs) if ins.engine == e):
                r = res.recs[res.recs["dep"] == d]
                assert np.array_equal(r["eng_thr"], r["sem_thr"]), (seed, d)
                checked += len(r)
    assert checked > 200


def test_hazard_catches_dropped_dependencies():
    w = chain_workload(seed=0)
    trips, off = w.trips.flat()
    for drop in range(len(w.prog.deps)):
        p = copy.deepcopy(w.prog)
        del p.deps[drop]
        res = core.run(p, trips, off[0], 0)
        assert hazard.check(p, res) != [], w.prog.deps[drop]


def test_hazard_catches_threshold_one_short():
    """Each dependency of the chain program is tight somewhere: for every one
    there is a consumer instance at which waiting for one retirement fewer than
    Eq. (1) requires leaves a race on the ring."""
    w = chain_workload(seed=0)
    trips, off = w.trips.flat()
    res = core.run(w.prog, trips, off[0], 0)
    for d in range(len(w.prog.deps)):
        idx = np.where((res.recs["dep"] == d) & (res.recs["sem_thr"] > 0))[0]
        found = False
        for i in idx:
            thr = res.recs["sem_thr"].copy()
            thr[i] -= 1
            if hazard.check(w.prog, res, thresholds=thr):
                found = True
                break
        assert found, w.prog.deps[d]


# --------------------------------------------------------------------------
# inputs and plain-math references
# --------------------------------------------------------------------------
def test_zipf_counts():
    c = zipf_counts(32768, 64, 1.1)
    assert c.sum() == 32768
    assert c[:5].tolist() == [8208, 3829, 2451, 1786, 1398]
    assert c[-3:].tolist() == [88, 86, 85]


def test_bf16_rounding():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9, -2.5, 3.0e38], np.float32)
    back = bf16_to_f32(to_bf16_bits(x))
    assert back.tolist()[:4] == [1.0, 1.0, 1.0 + 2 ** -7, -2.5]
    assert np.isfinite(back[4])


def test_gelu_values():
    g = mathref.gelu(np.array([0.0, 1.0, -1.0, 8.0, -8.0]))
    assert abs(g[0]) == 0.0
    assert abs(g[1] - 0.8413447460685429) < 1e-15
    assert abs(g[2] + 0.15865525393145707) < 1e-15
    assert abs(g[3] - 8.0) < 1e-12 and abs(g[4]) < 1e-12


def test_gemm_reference_special_cases():
    gi = gemm_inputs(seed=0, m=64, n=96, k=64)
    eye = to_bf16_bits(np.eye(96, 64, dtype=np.float32))          # B = I (first 64 cols)
    c = mathref.gemm_bias_gelu(gi.a, eye, gi.bias)
    a = bf16_to_f32(gi.a).astype(np.float64)
    assert np.allclose(c[:, :64], mathref.gelu(a + gi.bias[None, :64]), atol=1e-14)
    assert np.allclose(c[:, 64:], mathref.gelu(np.broadcast_to(gi.bias[64:], (64, 32))), atol=1e-14)
    rows, cols = np.array([0, 5, 63]), np.array([1, 70, 95])
    full = mathref.gemm_bias_gelu(gi.a, gi.bt, gi.bias)
    assert np.allclose(mathref.gemm_bias_gelu_at(gi.a, gi.bt, gi.bias, rows, cols), full[rows, cols])


def test_attention_reference_special_cases():
    ai = attn_inputs(seed=0, batch=2, heads=2, dim=16, lmin=5, lmax=9)
    scale = 0.25
    full = mathref.attention(ai.q, ai.k, ai.v, ai.cu_seqlens, scale)
    # constant V gives that constant
    v1 = to_bf16_bits(np.full(ai.v.shape, 0.75, np.float32))
    c = mathref.attention(ai.q, ai.k, v1, ai.cu_seqlens, scale)
    assert np.allclose(c, 0.75, atol=1e-14)
    # a single key returns its value
    one = attn_inputs(seed=1, batch=1, heads=1, dim=8, lengths=[1])
    o = mathref.attention(one.q, one.k, one.v, one.cu_seqlens, scale)
    assert np.allclose(o[0, 0], bf16_to_f32(one.v[0, 0]))
    # rows agree with the full evaluation
    rows = mathref.attention_rows(ai.q, ai.k, ai.v, ai.cu_seqlens, scale, [(1, 1, 2), (0, 0, 0)])
    s0 = ai.cu_seqlens[1]
    assert np.allclose(rows[0], full[s0 + 2, 1]) and np.allclose(rows[1], full[0, 0])


def test_attention_softmax_weights_closed_form():
    """Softmax weights pinned on scores with known exponentials: with scale
    1/2, query e_0 and keys 0, 2 e_0, -2 e_0 the scores are 0, 1, -1, so with
    V rows e_0, e_1, e_2 the output row is the softmax of (0, 1, -1) itself:
    (1, e, 1/e) / (1 + e + 1/e).  The first two keys alone give the logistic
    values 1/(1+e) and e/(1+e).  A zero query weights every key equally.
    A wrong exponent base, a dropped or doubled scale, or a transposed Q K
    product fails one of these."""
    d, scale = 4, 0.5
    q = np.zeros((3, 1, d), np.float32)
    q[0, 0, 0] = 1.0                                   # row 0: e_0; rows 1, 2: zero
    k = np.zeros((3, 1, d), np.float32)
    k[1, 0, 0], k[2, 0, 0] = 2.0, -2.0
    v = np.zeros((3, 1, d), np.float32)
    v[0, 0, 0], v[1, 0, 1], v[2, 0, 2] = 1.0, 1.0, 1.0
    q, k, v = (to_bf16_bits(a) for a in (q, k, v))
    # softmax(0, 1, -1) = (0.24472847105479764, 0.6652409557748219, 0.09003057317038046)
    want3 = np.array([0.24472847105479764, 0.6652409557748219, 0.09003057317038046, 0.0])
    cu3 = np.array([0, 3])
    full = mathref.attention(q, k, v, cu3, scale)
    assert np.abs(full[0, 0] - want3).max() < 1e-12
    assert np.abs(full[1, 0] - np.array([1 / 3, 1 / 3, 1 / 3, 0.0])).max() < 1e-12
    rows = mathref.attention_rows(q, k, v, cu3, scale, [(0, 0, 0), (0, 0, 2)])
    assert np.abs(rows[0] - want3).max() < 1e-12
    assert np.abs(rows[1] - np.array([1 / 3, 1 / 3, 1 / 3, 0.0])).max() < 1e-12
    # two keys: scores 0 and 1 give the logistic values 1/(1+e), e/(1+e)
    want2 = np.array([0.2689414213699951, 0.7310585786300049, 0.0, 0.0])
    cu2 = np.array([0, 2])
    two = mathref.attention(q[:2], k[:2], v[:2], cu2, scale)
    assert np.abs(two[0, 0] - want2).max() < 1e-12
    assert np.abs(mathref.attention_rows(q[:2], k[:2], v[:2], cu2, scale, [(0, 0, 0)])[0] - want2).max() < 1e-12


def test_moe_reference_properties():
    m = moe_inputs(seed=0, tokens=256, experts=4, hidden=32, ffn=16)
    assert m.counts.sum() == 256 and np.array_equal(np.bincount(m.assign, minlength=4), m.counts)
    assert (np.diff(m.assign[m.perm]) >= 0).all()
    y = mathref.moe_tokens(m, [0, 1, 2])
    # doubling W_down doubles the output; SiLU(0) = 0
    e = int(m.assign[0])
    wg, wu, wd = (bf16_to_f32(w).astype(np.float64) for w in m.weights(e))
    y2 = mathref.moe_tokens(m, [0], weights={e: (wg, wu, 2 * wd)})
    assert np.allclose(y2[0], 2 * y[0])
    y0 = mathref.moe_tokens(m, [0], weights={e: (0 * wg, wu, wd)})
    assert np.allclose(y0, 0)
    assert mathref.silu(np.array([0.0]))[0] == 0.0
    # SiLU(1) = 1 / (1 + e^-1) = 0.7310585786300049 (known constant)
    assert abs(mathref.silu(np.array([1.0]))[0] - 0.7310585786300049) < 1e-15
    # the hidden rows: with W_gate = W_up = I they are SiLU(x) * x, and the
    # full output is W_down applied to them
    eye = np.eye(16, 32)
    h = mathref.moe_hidden(m, [0], weights={e: (eye, eye, wd)})
    x = bf16_to_f32(m.x[0]).astype(np.float64)[:16]
    assert np.allclose(h[0], x * x / (1.0 + np.exp(-x)))
    assert np.allclose(mathref.moe_tokens(m, [0, 1]), [wd_e @ h_e for wd_e, h_e in zip(
        [(bf16_to_f32(m.weights(int(m.assign[t]))[2]).astype(np.float64)) for t in (0, 1)],
        mathref.moe_hidden(m, [0, 1]))])
