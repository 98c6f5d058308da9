"""Seeded synthetic workloads: programs, trip tables and input tensors.

Every random draw comes from ``numpy.random.default_rng(SeedSequence([cfg_id,
seed, wg]))`` (PCG64); "uniform [a, b]" on integers is inclusive.  Nothing in
this module computes a threshold, a loop register or a counter: it only lays
out the loop nest, the dependency graph, the per-execution trip counts and the
data that both the CPU oracle and the GPU library read.

Trip tables.  ``trips[loop][j]`` is the trip count of the j-th execution of the
loop statement ``loop`` inside one workgroup (a loop statement executes once
per iteration of its parent, so j runs over all parent iterations in order).
The flat form is ``trips`` (int32, concatenated) plus ``trip_off`` (int64
``[n_wg][n_loops]``) giving where each loop's list starts; the top-level loop
has a single entry 1.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .program import (OP_ADDC, OP_MOE_EPI, OP_MOE_LOAD, OP_MOE_MMA, OP_MOE_SPILL, OP_ATTN_LOAD, OP_ATTN_NORM, OP_ATTN_PREAD, OP_ATTN_PV, OP_ATTN_QK, OP_ATTN_SM,
                      OP_GEMM_BIAS, OP_GEMM_EPI, OP_GEMM_LOAD, OP_GEMM_MMA,
                      OP_GEMM_SPILL, OP_LOAD, OP_NOP, OP_SCALE_ACC, OP_STORE_ACC,
                      OP_ADAM_LOAD, OP_ADAM_STORE, OP_ADAM_UPDATE, OP_RMS_LOAD, OP_RMS_NORM, OP_RMS_STORE,
                      OP_STORE_RING, Program, ProgramBuilder,
                      f32_bits, tile_args)

CFG_CHAIN, CFG_STREAM, CFG_GEMM, CFG_ATTN, CFG_MOE, CFG_RANDOM = 1, 2, 3, 4, 5, 99
CFG_LAG = 6
CFG_RMS = 7
CFG_ADAM = 8


def rng_for(cfg_id: int, seed: int, wg: int = 0) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([cfg_id, seed, wg]))


# ---------------------------------------------------------------------------
# trip tables
# ---------------------------------------------------------------------------
@dataclass
class TripTables:
    per_wg: list          # per workgroup: list over loops of np.int32 arrays

    @property
    def n_wg(self) -> int:
        return len(self.per_wg)

    def flat(self):
        n_loops = len(self.per_wg[0])
        off = np.zeros((self.n_wg, n_loops), dtype=np.int64)
        chunks, pos = [], 0
        for w, loops in enumerate(self.per_wg):
            for l, arr in enumerate(loops):
                off[w, l] = pos
                chunks.append(np.asarray(arr, dtype=np.int32))
                pos += len(arr)
        trips = np.concatenate(chunks) if chunks else np.zeros(0, np.int32)
        return trips.astype(np.int32), off

    def total_iters(self, wg: int, loop: int) -> int:
        return int(np.sum(self.per_wg[wg][loop], dtype=np.int64))


def draw_trips(prog: Program, draw) -> list:
    """Trip lists for one workgroup.  ``draw(loop, n_exec)`` returns the trip
    counts of the ``n_exec`` executions of ``loop``.  Loops are numbered so
    that a parent precedes its children, so one pass suffices."""
    trips = [np.array([1], dtype=np.int32)]
    for l in range(1, prog.n_loops):
        parent = prog.loop_parent[l]
        n_exec = int(np.sum(trips[parent], dtype=np.int64))
        t = np.asarray(draw(l, n_exec), dtype=np.int32)
        assert t.shape == (n_exec,)
        trips.append(t)
    return trips


def tile_bases(tt: TripTables, loop: int) -> np.ndarray:
    """Exclusive prefix sum over workgroups of the iteration count of ``loop``:
    workgroup w's tiles start at this index in the packed tile buffers."""
    counts = np.array([tt.total_iters(w, loop) for w in range(tt.n_wg)], dtype=np.int64)
    return np.concatenate([[0], np.cumsum(counts)[:-1]]).astype(np.int64), counts


# ---------------------------------------------------------------------------
# cfg1: 2-engine chain, one workgroup
# ---------------------------------------------------------------------------
def chain_program(ring_slots: int = 4, scale: float = 0.5, kernel: str = "chain") -> Program:
    """E0 loads 256-element fp32 tiles into a ring, E1 accumulates 0.5 * tile.

    A{ E0:ACQ; B{ E0:LOAD X[n] -> ring[(rhat_B-1) % 4]; E1:CONS acc += 0.5*ring }}
    E1:STORE acc -> out

    LOAD->CONS (k=0) is the read-after-write; CONS->LOAD (k=4) keeps a slot
    from being refilled before it is read within one trip of B; CONS->ACQ
    (k=1) orders the next trip's loads after the previous trip's reads.
    ``kernel``: "chain" (the dedicated two-wave kernel) or "interp" (the
    generic interpreter)."""
    b = ProgramBuilder(kernel, n_engines=2)
    with b.loop("A") as A:
        b.instr(0, OP_NOP, name="ACQ")
        with b.loop("B") as B:
            b.instr(0, OP_LOAD, tile_args(src=1, dst=0, pos_loop=B, per_gen=ring_slots, idx_loop=B),
                    name="LOAD")
            b.instr(1, OP_SCALE_ACC, tile_args(src=0, dst=0, pos_loop=B, per_gen=ring_slots, const=scale),
                    name="CONS")
    b.instr(1, OP_STORE_ACC, tile_args(src=0, dst=2), name="STORE")
    b.dep("LOAD", "CONS", 0)
    b.dep("CONS", "LOAD", ring_slots)
    b.dep("CONS", "ACQ", 1)
    p = b.build()
    p.tile_elems = 256
    p.ring_slots = [ring_slots]
    p.n_accs = 1
    return p


@dataclass
class ChainWorkload:
    prog: Program
    trips: TripTables
    base: np.ndarray      # int64 [n_wg]: tile base per workgroup
    x: np.ndarray         # fp32 [n_tiles, 256]
    n_tiles: int


def chain_workload(seed: int = 0, outer: int = 16, inner_max: int = 8, n_wg: int = 1,
                   kernel: str = "chain", ring_slots: int = 4) -> ChainWorkload:
    prog = chain_program(ring_slots=ring_slots, kernel=kernel)
    per = []
    for w in range(n_wg):
        rng = rng_for(CFG_CHAIN, seed, w)

        def draw(l, n, rng=rng):
            if l == 1:
                return np.full(n, outer)
            return rng.integers(1, inner_max + 1, size=n)
        per.append(draw_trips(prog, draw))
    tt = TripTables(per)
    base, counts = tile_bases(tt, prog.loop_id("B"))
    n_tiles = int(counts.sum())
    xs = [rng_for(CFG_CHAIN, seed, 1000 + w).uniform(-1.0, 1.0, size=(int(counts[w]), 256)).astype(np.float32)
          for w in range(n_wg)]
    return ChainWorkload(prog, tt, base, np.concatenate(xs), n_tiles)


# ---------------------------------------------------------------------------
# A software pipeline whose dependencies need the barrier fallback
# ---------------------------------------------------------------------------
def lag_pipeline_program(lag: int = 2, ring_slots: int = 3, scale: float = 0.5) -> Program:
    """Two-stage pipeline: the tile loaded in iteration o of O is consumed in
    iteration o + lag (a prologue of ``lag`` iterations skips the consumer).

      O{ C(cond: trip 1 once O has run lag iterations){ E1:CONS acc += 0.5*ring[(r_C-1) % R] }
         M(cond: trip 1){ E0:LOAD X[r_M-1] -> ring[(r_M-1) % R] } }
      E1:STORE acc -> out

    Inside C, r_C = r_O - lag and r_M = r_O, so CONS reads the slot LOAD
    filled lag iterations of O earlier.  LOAD->CONS (offset lag, backward:
    C precedes M in O's body) and CONS->LOAD (offset R - lag, forward: the
    slot's previous reader ran R - lag iterations earlier) both have the
    producer nested below O, so for lag >= 2 and R - lag >= 1 neither is one
    of the allocatable cases of Section 5.2; CONS->STORE (offset 0 at the top
    level, producer nested, forward) is.  Output: 0.5 * (sum of the first
    trip(O) - lag tiles)."""
    assert 1 <= lag < ring_slots
    b = ProgramBuilder("interp", n_engines=2)
    with b.loop("O"):
        with b.loop("C", is_cond=True) as C:
            b.instr(1, OP_SCALE_ACC, tile_args(src=0, dst=0, gen_loop=C, n_gen=ring_slots, const=scale),
                    name="CONS")
        with b.loop("M", is_cond=True) as M:
            b.instr(0, OP_LOAD, tile_args(src=1, dst=0, gen_loop=M, n_gen=ring_slots, idx_loop=M),
                    name="LOAD")
    b.instr(1, OP_STORE_ACC, tile_args(src=0, dst=2), name="STORE")
    b.dep("LOAD", "CONS", lag)
    b.dep("CONS", "LOAD", ring_slots - lag)
    b.dep("CONS", "STORE", 0)
    p = b.build()
    p.tile_elems = 256
    p.ring_slots = [ring_slots]
    p.n_accs = 1
    return p


def lag_pipeline_workload(seed: int = 0, n_wg: int = 1, outer_min: int = 1, outer_max: int = 24, lag: int = 2,
                          ring_slots: int = 3) -> ChainWorkload:
    """Per workgroup a trip of O drawn from [outer_min, outer_max] (trips
    below lag + 1 never consume); X ~ U(-1, 1) fp32 tiles of 256."""
    prog = lag_pipeline_program(lag, ring_slots)
    O, C, M = prog.loop_id("O"), prog.loop_id("C"), prog.loop_id("M")
    per = []
    for w in range(n_wg):
        rng = rng_for(CFG_LAG, seed, w)
        outer = int(rng.integers(outer_min, outer_max + 1))

        def draw(l, n, outer=outer):
            if l == O:
                return np.full(n, outer)
            if l == C:
                return (np.arange(1, n + 1) > lag).astype(np.int32)
            return np.ones(n, np.int32)
        per.append(draw_trips(prog, draw))
    tt = TripTables(per)
    base, counts = tile_bases(tt, M)
    xs = [rng_for(CFG_LAG, seed, 1000 + w).uniform(-1.0, 1.0, size=(int(counts[w]), 256)).astype(np.float32)
          for w in range(n_wg)]
    return ChainWorkload(prog, tt, base, np.concatenate(xs), int(counts.sum()))


# ---------------------------------------------------------------------------
# A ring indexed across trips (linearized-offset extension)
# ---------------------------------------------------------------------------
def ring_program(ring_slots: int = 4, scale: float = 0.5, linear: bool = True) -> Program:
    """The chain's two engines with the ring slot taken from the monotone
    register of B, so that slots rotate across trips of B:

      A{ [E0:ACQ] B{ E0:LOAD X[r_B-1] -> ring[(r_B-1) % R]; E1:CONS acc += 0.5*ring[(r_B-1) % R] } }
      E1:STORE acc -> out

    ``linear=True``: CONS->LOAD at offset R with the linearized reading (an
    extension, not in the paper) orders every slot reuse, also the ones that
    straddle a trip boundary, with one dependency and no ACQ.
    ``linear=False``: the paper's relation: CONS->LOAD at offset R underflows
    in the first R iterations of every trip, so an ACQ instruction with
    CONS->ACQ at offset 1 (C3) drains the previous trip's reads at each trip
    start."""
    b = ProgramBuilder("interp", n_engines=2)
    with b.loop("A"):
        if not linear:
            b.instr(0, OP_NOP, name="ACQ")
        with b.loop("B") as B:
            slot = dict(gen_loop=B, n_gen=ring_slots)
            b.instr(0, OP_LOAD, tile_args(src=1, dst=0, idx_loop=B, **slot), name="LOAD")
            b.instr(1, OP_SCALE_ACC, tile_args(src=0, dst=0, const=scale, **slot), name="CONS")
    b.instr(1, OP_STORE_ACC, tile_args(src=0, dst=2), name="STORE")
    b.dep("LOAD", "CONS", 0)
    b.dep("CONS", "LOAD", ring_slots, linear=linear)
    if not linear:
        b.dep("CONS", "ACQ", 1)
    b.dep("CONS", "STORE", 0)
    p = b.build()
    p.tile_elems = 256
    p.ring_slots = [ring_slots]
    p.n_accs = 1
    return p


def ring_workload(seed: int = 0, outer: int = 16, inner_max: int = 8, n_wg: int = 1, ring_slots: int = 4,
                  linear: bool = True) -> ChainWorkload:
    """The chain's trip recipe (outer trip fixed, inner trips U[1, inner_max]
    per workgroup) on the ring program."""
    prog = ring_program(ring_slots, linear=linear)
    A, B = prog.loop_id("A"), prog.loop_id("B")
    per = []
    for w in range(n_wg):
        rng = rng_for(CFG_CHAIN, seed, w)

        def draw(l, n, rng=rng):
            if l == A:
                return np.full(n, outer)
            return rng.integers(1, inner_max + 1, size=n)
        per.append(draw_trips(prog, draw))
    tt = TripTables(per)
    base, counts = tile_bases(tt, B)
    xs = [rng_for(CFG_CHAIN, seed, 1000 + w).uniform(-1.0, 1.0, size=(int(counts[w]), 256)).astype(np.float32)
          for w in range(n_wg)]
    return ChainWorkload(prog, tt, base, np.concatenate(xs), int(counts.sum()))


# ---------------------------------------------------------------------------
# cfg2: sync-bound 3-engine stream, 1024 workgroups
# ---------------------------------------------------------------------------
STREAM_GENERATIONS = 32   # ring generations of the in-place layout (>= twice the largest M trip)


def stream_program(n_gen: int = STREAM_GENERATIONS, per_gen: int = 4, inner_war: bool = False,
                   layout: str = "inplace") -> Program:
    """Load / vector-add / store engines over a 3-level nest O{M{I{...}}}.

    Ring slot = ((r_M - 1) % n_gen) * per_gen + (rhat_I - 1): each M iteration
    owns one generation of per_gen slots.  With inner trips of at most per_gen
    a slot is never reused inside one trip of I; ``inner_war`` adds the
    offset-per_gen dependencies that would order such reuse.

    ``layout="inplace"`` (default): one ring; the add engine rewrites the slot
    in place and the store engine reads it back:

      O{ E0:ACQ_O  M{ I{ E0:LOAD X->r[slot]  E1:ADD r[slot]+1->r[slot]  E2:STORE r[slot]->Y } }  E2:MARK_O }

    With M trips of at most n_gen / 2, the generations of two consecutive O
    iterations are disjoint, so MARK_O -> ACQ_O at offset 2 (the store engine
    has finished O iteration o - 2) orders every slot reuse and no M-level
    instruction is needed: the load engine may run a whole O iteration ahead.

    ``layout="two_rings"``: rings X (load -> add) and Y (add -> store) with
    acquire / marker instructions at M (offset n_gen) and O (offset 1):

      O{ E0:ACQX_O E1:ACQY_O
         M{ E0:ACQX_M E1:ACQY_M
            I{ E0:LOAD X->rx[slot]  E1:ADD rx[slot]+1->ry[slot]  E2:STORE ry[slot]->Y }
            E1:MARKX_M E2:MARKY_M }
         E1:MARKX_O E2:MARKY_O }
    """
    b = ProgramBuilder("stream3", n_engines=3)
    if layout == "inplace":
        with b.loop("O"):
            b.instr(0, OP_NOP, name="ACQ_O")
            with b.loop("M") as M:
                with b.loop("I") as I:
                    slot = dict(gen_loop=M, n_gen=n_gen, pos_loop=I, per_gen=per_gen)
                    b.instr(0, OP_LOAD, tile_args(src=1, dst=0, idx_loop=I, **slot), name="LOAD")
                    b.instr(1, OP_ADDC, tile_args(src=0, dst=0, const=1.0, **slot), name="ADD")
                    b.instr(2, OP_STORE_RING, tile_args(src=0, dst=2, idx_loop=I, **slot), name="STORE")
            b.instr(2, OP_NOP, name="MARK_O")
        b.dep("LOAD", "ADD", 0)
        b.dep("ADD", "STORE", 0)
        if inner_war:
            b.dep("STORE", "LOAD", per_gen)
        b.dep("MARK_O", "ACQ_O", 2)
        p = b.build()
        p.tile_elems = 64
        p.ring_slots = [n_gen * per_gen]
        return p
    if layout != "two_rings":
        raise ValueError(layout)
    with b.loop("O"):
        b.instr(0, OP_NOP, name="ACQX_O")
        b.instr(1, OP_NOP, name="ACQY_O")
        with b.loop("M") as M:
            b.instr(0, OP_NOP, name="ACQX_M")
            b.instr(1, OP_NOP, name="ACQY_M")
            with b.loop("I") as I:
                slot = dict(gen_loop=M, n_gen=n_gen, pos_loop=I, per_gen=per_gen)
                b.instr(0, OP_LOAD, tile_args(src=1, dst=0, idx_loop=I, **slot), name="LOAD")
                b.instr(1, OP_ADDC, tile_args(src=0, dst=1, const=1.0, **slot), name="ADD")
                b.instr(2, OP_STORE_RING, tile_args(src=1, dst=2, idx_loop=I, **slot), name="STORE")
            b.instr(1, OP_NOP, name="MARKX_M")
            b.instr(2, OP_NOP, name="MARKY_M")
        b.instr(1, OP_NOP, name="MARKX_O")
        b.instr(2, OP_NOP, name="MARKY_O")
    b.dep("LOAD", "ADD", 0)
    b.dep("ADD", "STORE", 0)
    if inner_war:
        # slot reuse inside one trip of I; never owed when inner trips are at
        # most per_gen (the hazard check proves the program covered without it)
        b.dep("ADD", "LOAD", per_gen)
        b.dep("STORE", "ADD", per_gen)
    b.dep("MARKX_M", "ACQX_M", n_gen)    # generation reuse across M iterations
    b.dep("MARKY_M", "ACQY_M", n_gen)
    b.dep("MARKX_O", "ACQX_O", 1)        # across O iterations
    b.dep("MARKY_O", "ACQY_O", 1)
    p = b.build()
    p.tile_elems = 64
    p.ring_slots = [n_gen * per_gen, n_gen * per_gen]
    return p


@dataclass
class StreamWorkload:
    prog: Program
    trips: TripTables
    base: np.ndarray      # int64 [n_wg]
    counts: np.ndarray    # int64 [n_wg]: inner iterations per workgroup
    x: np.ndarray | None  # fp32 [n_tiles, 64]
    n_tiles: int


def stream_workload(seed: int = 0, n_wg: int = 1024, outer: int = 256, mid_max: int = 16,
                    inner_max: int = 4, n_gen: int = STREAM_GENERATIONS, with_data: bool = True,
                    inner_war: bool = False, layout: str = "inplace") -> StreamWorkload:
    if layout == "inplace" and n_gen < 2 * mid_max:
        raise ValueError("the in-place layout needs at least twice the largest M trip in generations")
    prog = stream_program(n_gen=n_gen, per_gen=inner_max, inner_war=inner_war, layout=layout)
    per = []
    for w in range(n_wg):
        rng = rng_for(CFG_STREAM, seed, w)

        def draw(l, n, rng=rng):
            if l == 1:
                return np.full(n, outer)
            if l == 2:
                return rng.integers(1, mid_max + 1, size=n)
            return rng.integers(1, inner_max + 1, size=n)
        per.append(draw_trips(prog, draw))
    tt = TripTables(per)
    base, counts = tile_bases(tt, prog.loop_id("I"))
    n_tiles = int(counts.sum())
    x = None
    if with_data:
        x = np.empty((n_tiles, 64), dtype=np.float32)
        for w in range(n_wg):
            g = rng_for(CFG_STREAM, seed, 100000 + w)
            x[base[w]:base[w] + counts[w]] = g.uniform(-1.0, 1.0, size=(int(counts[w]), 64))
    return StreamWorkload(prog, tt, base, counts, x, n_tiles)


def stream_fixed_trips(prog: Program, m_trips, i_trip: int, n_wg: int = 1) -> TripTables:
    """Trip tables of one or more identical workgroups: O runs len(m_trips)
    iterations with those M trips, every trip of I is i_trip."""
    m_trips = np.asarray(m_trips, dtype=np.int32)

    def draw(l, n):
        if l == 1:
            return np.full(n, len(m_trips))
        if l == 2:
            return m_trips[:n]
        return np.full(n, i_trip)
    return TripTables([draw_trips(prog, draw) for _ in range(n_wg)])


# ---------------------------------------------------------------------------
# random tiny nests (property tests of thresholds)
# ---------------------------------------------------------------------------
def random_nest(seed: int, max_depth: int = 3, n_engines: int = 3, max_items: int = 3,
                max_trip: int = 3, n_deps: int = 6, max_k: int = 3):
    """A random structured program with random dependency triples.

    Offsets are drawn uniformly from [0, max_k], so some triples fall outside
    the allocatable subset; callers keep whichever the planner accepts.
    Returns (program, trip tables for one workgroup)."""
    rng = rng_for(CFG_RANDOM, seed)
    b = ProgramBuilder("interp", n_engines=n_engines)

    def fill(depth):
        n_items = int(rng.integers(1, max_items + 1))
        for _ in range(n_items):
            if depth < max_depth and rng.random() < 0.45:
                with b.loop(f"L{len(b.p.loop_parent)}", is_cond=bool(rng.random() < 0.2)):
                    fill(depth + 1)
            else:
                for _ in range(int(rng.integers(1, 4))):
                    b.instr(int(rng.integers(0, n_engines)), OP_NOP)
                b.block_break() if rng.random() < 0.3 else None

    fill(0)
    if not b.p.instrs:
        b.instr(0, OP_NOP)
    n_ins = len(b.p.instrs)
    for _ in range(n_deps):
        pr, cn = (int(v) for v in rng.integers(0, n_ins, size=2))
        if pr == cn:
            continue
        b.dep(pr, cn, int(rng.integers(0, max_k + 1)))
    prog = b.build()

    def draw(l, n):
        hi = 1 if prog.loop_is_cond[l] else max_trip
        return rng.integers(0, hi + 1, size=n)
    tt = TripTables([draw_trips(prog, draw)])
    return prog, tt


# ---------------------------------------------------------------------------
# cfg3: GEMM + bias + GELU with load / MFMA / epilogue engines
# ---------------------------------------------------------------------------
GEMM_TILE = 256     # output tile edge per workgroup
GEMM_BK = 32        # K step per ring slot
GEMM_RING = 4       # ring slots of the K loop
GEMM_E_RING = 4     # epilogue slots (in the K ring's memory after the K loop; 4 measured 1 % faster than 2, as fast as 8)
GEMM_CHUNKS = 8     # accumulator blocks spilled per MFMA wave


def gemm_program(m: int, n: int, k: int, ring: int = GEMM_RING, e_ring: int = GEMM_E_RING,
                 load_waves: int = 2, mma_waves: int = 8, epi_waves: int = 2) -> Program:
    """One 256 x 256 output tile per workgroup:

      E0: BIAS
      K{ E0: LOAD A, B tiles of the step -> ring[(rhat_K - 1) % ring]; E1: MMA }
      C{ E1: SPILL bias + GELU of one accumulator block -> ering[(rhat_C - 1) % e_ring]; E2: EPI store }

    LOAD->MMA (k=0) and MMA->LOAD (k=ring) protect the K ring, SPILL->EPI
    (k=0) and EPI->SPILL (k=e_ring) the epilogue ring, BIAS->SPILL (k=0 at the
    top level) the staged bias.  The epilogue ring occupies the memory of the
    K ring, so MMA->SPILL (k=0; producer nested in K, consumer in C) lets a
    spill start only after every MFMA wave retired its last K step."""
    b = ProgramBuilder("gemm", n_engines=3, waves_per_engine=[load_waves, mma_waves, epi_waves])
    b.instr(0, OP_GEMM_BIAS, [m, n, k, 0, 0, 0, 0, 0], name="BIAS")
    with b.loop("K"):
        b.instr(0, OP_GEMM_LOAD, [m, n, k, ring, 0, 0, 0, 0], name="LOAD")
        b.instr(1, OP_GEMM_MMA, [0] * 8, name="MMA")
    with b.loop("C"):
        b.instr(1, OP_GEMM_SPILL, [e_ring, 0, 0, 0, 0, 0, 0, 0], name="SPILL")
        b.instr(2, OP_GEMM_EPI, [0] * 8, name="EPI")
    b.dep("LOAD", "MMA", 0)
    b.dep("MMA", "LOAD", ring)
    b.dep("BIAS", "SPILL", 0)
    b.dep("SPILL", "EPI", 0)
    b.dep("EPI", "SPILL", e_ring)
    b.dep("MMA", "SPILL", 0)
    return b.build()


GEMM_K_UNROLLED_STEPS = (3, 8, 128)   # K steps the K-unrolled kernel is built for


def gemm_program_k_unrolled(m: int, n: int, k: int, ring: int = GEMM_RING, e_ring: int = GEMM_E_RING) -> Program:
    """The GEMM with its K loop removed (the K-unrolled variant of the
    paper's tiled matmul): the K / 32 steps are listed one after another at
    the top level, so every threshold of the K phase is a static ordinal:

      E0: BIAS
      E0: LOAD_0  E1: MMA_0  E0: LOAD_1  E1: MMA_1 ...  (step s in slot s % ring)
      C{ E1: SPILL; E2: EPI }

    LOAD_s->MMA_s and MMA_s->LOAD_{s+ring} at offset 0 (forward in the
    straight line), BIAS->SPILL, MMA_last->SPILL (every MFMA wave has
    retired its last step before the epilogue reuses the ring's memory;
    retirement is in order), SPILL->EPI, EPI->SPILL as in gemm_program."""
    steps = k // GEMM_BK
    b = ProgramBuilder("gemm", n_engines=3, waves_per_engine=[2, 8, 2])
    b.instr(0, OP_GEMM_BIAS, [m, n, k, 0, 0, 0, 0, 0], name="BIAS")
    for st in range(steps):
        b.instr(0, OP_GEMM_LOAD, [m, n, k, ring, st, 0, 0, 0], name=f"LOAD{st}")
        b.instr(1, OP_GEMM_MMA, [st, 0, 0, 0, 0, 0, 0, 0], name=f"MMA{st}")
    with b.loop("C"):
        b.instr(1, OP_GEMM_SPILL, [e_ring, 0, 0, 0, 0, 0, 0, 0], name="SPILL")
        b.instr(2, OP_GEMM_EPI, [0] * 8, name="EPI")
    for st in range(steps):
        b.dep(f"LOAD{st}", f"MMA{st}", 0)
        if st + ring < steps:
            b.dep(f"MMA{st}", f"LOAD{st + ring}", 0)
    b.dep("BIAS", "SPILL", 0)
    b.dep("SPILL", "EPI", 0)
    b.dep("EPI", "SPILL", e_ring)
    b.dep(f"MMA{steps - 1}", "SPILL", 0)
    return b.build()


def gemm_trips_k_unrolled(m: int, n: int) -> TripTables:
    """The K-unrolled GEMM's trip tables: the epilogue loop's 8 chunks."""
    n_wg = (m // GEMM_TILE) * (n // GEMM_TILE)
    return TripTables([[np.array([1], np.int32), np.array([GEMM_CHUNKS], np.int32)] for _ in range(n_wg)])


def gemm_trips(m: int, n: int, k: int, ring: int = GEMM_RING) -> TripTables:
    """Every workgroup runs the K loop once with K / 32 steps and the
    epilogue loop once with 8 chunks."""
    n_wg = (m // GEMM_TILE) * (n // GEMM_TILE)
    one = [np.array([1], np.int32), np.array([k // GEMM_BK], np.int32), np.array([GEMM_CHUNKS], np.int32)]
    return TripTables([[a.copy() for a in one] for _ in range(n_wg)])


# ---------------------------------------------------------------------------
# cfg4: variable-length attention forward with K load / QK^T / softmax / PV /
# V load engines
# ---------------------------------------------------------------------------
ATTN_BQ = 128       # query rows per workgroup
ATTN_BKV = 64       # keys per KV block
ATTN_D = 128        # head dimension
ATTN_SP = 2         # S/P buffer slots
ATTN_NK = 2         # K ring slots of the benchmark layout
ATTN_NV = 3         # V ring slots of the benchmark layout (2 + 3 measured 2 % faster than 3 + 2)
ATTN_LINEAR = False # benchmark form: the paper's relation with acquires at each tile (True: linearized reuse)


def attn_program(heads: int, dim: int = ATTN_D, nk: int = ATTN_NK, nv: int = ATTN_NV,
                 linear: bool = ATTN_LINEAR) -> Program:
    """A fixed set of workgroups, each running a run-time list of (sequence,
    head, 128-query tile) work items:

      T{ E0: ACQK  E4: ACQV  E1: ACQS
         KV{ E0: LOADK K block -> kring[(r_KV - 1) % nk]
             E4: LOADV V block -> vring[(r_KV - 1) % nv]
             E1: QK    S = Q K^T -> sp[(r_KV - 1) % 2]
             E2: SM    online softmax: P over S in place, alpha, running sum l
             E3: PREAD P and alpha of the step into registers
             E3: PV    O = alpha O + P V }
         E3: NORM  O / l -> output }

    T's trip count is the workgroup's number of tiles, KV's ceil(L / 64) for
    the tile's sequence length L; both known only at run time.  LOADK->QK,
    LOADV->PV, QK->SM, SM->PREAD (k=0) carry the data forward.  The rings
    and S/P slots are indexed by r_KV, which counts KV iterations over all
    tiles.  Their reuse dependencies QK->LOADK (k=nk), PV->LOADV (k=nv) and
    PREAD->QK (k=2) are read per trip of KV (the paper's relation), and the
    acquire instructions at each tile with QK->ACQK, PV->ACQV, PREAD->ACQS
    (k=1, C3 at T) drain the previous tile's reads of the rings and S/P
    slots before the next tile refills them.  SM->NORM (k=0, C2) delivers a
    tile's final row sums; they are double-buffered by tile, and NORM->SM
    (k=2, C1 at T) keeps a tile's softmax from overwriting a buffer before
    NORM of the tile before last has read it.

    ``linear=True`` reads the three reuse dependencies with the linearized
    offset instead (an extension of the paper's relation) and drops the
    acquire instructions: the next tile's loads and QK steps overlap the end
    of the previous tile."""
    b = ProgramBuilder("attn", n_engines=5, waves_per_engine=[1, 2, 4, 4, 1])
    with b.loop("T"):
        if not linear:
            b.instr(0, OP_NOP, [0] * 8, name="ACQK")
            b.instr(4, OP_NOP, [0] * 8, name="ACQV")
            b.instr(1, OP_NOP, [0] * 8, name="ACQS")
        with b.loop("KV"):
            b.instr(0, OP_ATTN_LOAD, [0, nk, heads, dim, 0, 0, 0, 0], name="LOADK")
            b.instr(4, OP_ATTN_LOAD, [1, nv, heads, dim, 0, 0, 0, 0], name="LOADV")
            b.instr(1, OP_ATTN_QK, [0] * 8, name="QK")
            b.instr(2, OP_ATTN_SM, [0] * 8, name="SM")
            b.instr(3, OP_ATTN_PREAD, [0] * 8, name="PREAD")
            b.instr(3, OP_ATTN_PV, [0] * 8, name="PV")
        b.instr(3, OP_ATTN_NORM, [0] * 8, name="NORM")
    b.dep("LOADK", "QK", 0)
    b.dep("LOADV", "PV", 0)
    b.dep("QK", "SM", 0)
    b.dep("SM", "PREAD", 0)
    b.dep("QK", "LOADK", nk, linear=linear)
    b.dep("PV", "LOADV", nv, linear=linear)
    b.dep("PREAD", "QK", ATTN_SP, linear=linear)
    if not linear:
        b.dep("QK", "ACQK", 1)
        b.dep("PV", "ACQV", 1)
        b.dep("PREAD", "ACQS", 1)
    b.dep("SM", "NORM", 0)
    b.dep("NORM", "SM", 2)
    return b.build()


@dataclass
class AttnWork:
    work: np.ndarray      # int32 [max tiles * n_wg, 4]: first token, length, first query row, head;
                          # tile j of workgroup w at row w + j * n_wg
    trips: TripTables     # per workgroup: [[1], [tiles], [ceil(L / 64) per tile]]


ATTN_WG = 256                # workgroups: one per compute unit (the LDS allows one per CU)
ATTN_TILE_COST = 5           # fixed cost of a tile in KV steps, for balancing (measured on uniform
                             # lengths: about 6.3 us per tile against 1.27 us per KV step; 0, 5, 9
                             # and 14 time the same within 2 %)


def attn_worklist(lengths, heads: int, xcds: int = 8, n_wg: int = ATTN_WG) -> AttnWork:
    """Tiles (sequence, head, 128-query tile) assigned to ``n_wg``
    workgroups.

    (sequence, head) pairs are taken longest first and each goes, with all
    of its query tiles, to the XCD with the least work so far, so a pair's
    tiles share one L2 for their K and V blocks (workgroup w runs on XCD
    w % xcds).  Within an XCD, tiles in that order go to the workgroup with
    the least work so far (KV steps plus a fixed cost per tile), so the
    tiles of one pair run at the same time on different compute units."""
    if n_wg <= 0:
        raise ValueError("n_wg must be positive")
    lengths = np.asarray(lengths, dtype=np.int64)
    cu = np.concatenate([[0], np.cumsum(lengths)])
    pairs = sorted(((int(lengths[b]), b, h) for b in range(len(lengths)) for h in range(heads)),
                   key=lambda t: (-t[0], t[1], t[2]))
    load = [0] * xcds
    lists = [[] for _ in range(xcds)]
    for L, b, h in pairs:
        if L <= 0:
            continue
        x = min(range(xcds), key=lambda i: (load[i], i))
        n_tiles = -(-L // ATTN_BQ)
        load[x] += n_tiles * (-(-L // ATTN_BKV) + ATTN_TILE_COST)
        for t in range(n_tiles):
            lists[x].append((int(cu[b]), L, t * ATTN_BQ, h))
    per_wg = [[] for _ in range(n_wg)]
    wg_load = [0] * n_wg
    for x in range(xcds):
        mine = list(range(x, n_wg, xcds)) or list(range(n_wg))
        for item in lists[x]:
            w = min(mine, key=lambda i: (wg_load[i], i))
            per_wg[w].append(item)
            wg_load[w] += -(-item[1] // ATTN_BKV) + ATTN_TILE_COST
    depth = max((len(l) for l in per_wg), default=0)
    work = np.zeros((max(depth, 1) * n_wg, 4), np.int32)
    for w, items in enumerate(per_wg):
        for j, it in enumerate(items):
            work[w + j * n_wg] = it
    trips = TripTables([[np.array([1], np.int32), np.array([len(items)], np.int32),
                         np.array([-(-int(L) // ATTN_BKV) for _, L, _, _ in items], np.int32)]
                        for items in per_wg])
    return AttnWork(work, trips)


# ---------------------------------------------------------------------------
# cfg5: MoE grouped GEMM, two phases with load / MFMA / epilogue engines and a
# runtime M-tile loop per workgroup
# ---------------------------------------------------------------------------
MOE_BM = 256                 # token rows per M-tile (128 or 256)
MOE_BK = 32                  # K step per ring slot
MOE_BN = {1: 128, 2: 256}    # output columns per workgroup: h columns (phase 1), y columns (phase 2)
# (ring slots, epilogue slots) per M-tile height and phase: a ring slot
# holds BM x 64 B of token rows and 16 KiB of weight rows; with the 2 KiB of
# counters and 16 KiB epilogue slots they stay within 160 KiB of LDS.
# Epilogue slots 0: each chunk of an M-tile in its own 16 KiB of the ring,
# after the tile's K loop (four 32 KiB slots hold phase 2's eight chunks of
# a 256-row tile).  At 256 rows, in one process: phase 1 (4 chunks) 1-1.7 %
# faster in the ring than with one epilogue slot (1001 against 1011-1018 us;
# the other way round before the output stores were plain and the gather
# indices prefetched), phase 2 (8 chunks) 2-3 % faster in the ring than with
# three ring slots and one or two epilogue slots.
MOE_RINGS = {(128, 1): (5, 2), (128, 2): (5, 2), (256, 1): (4, 0), (256, 2): (4, 0)}
MOE_MCHUNKS = {128: 4, 256: 4}   # at most this many M-tiles per workgroup


def moe_chunks(phase: int, bm: int = MOE_BM) -> int:
    """Epilogue chunks per M-tile: one 32-row block of each MFMA wave's
    BM / 2-row sub-tile (phase 1), times its two 32-column blocks (phase 2)."""
    return bm // 64 * (1 if phase == 1 else 2)


MOE_LINEAR = False           # benchmark ring form: the paper's ACQL drain at every M-tile;
                             # True selects the linearized MMA->LOAD dependency (extension)


def moe_program(phase: int, hidden: int, ffn: int, ring: int = None, e_ring: int = None,
                linear: bool = MOE_LINEAR, bm: int = MOE_BM) -> Program:
    """One workgroup per (expert, N-tile, run of M-tiles); phase 1 computes
    h = SiLU(x W_gate) * (x W_up) for 128 h columns, phase 2 y = h W_down for
    256 y columns:

      M{ E0: ACQL
         K{ E0: LOAD token rows and weight rows of the step -> ring[(rhat_K - 1) % ring]; E1: MMA }
         E1: ACQE
         C{ E1: SPILL one accumulator block per MFMA wave -> epilogue slot; E2: EPI store } }

    The M loop's trip count is the number of ``bm``-token tiles (128 or
    256) of the workgroup's expert it covers, known only at run time;
    ``ring`` and ``e_ring`` default to what fits in LDS for that tile
    height.  LOAD->MMA (k=0) and MMA->LOAD (k=ring) protect the ring inside
    an M-tile, SPILL->EPI (k=0) hands over each chunk, EPI->ACQE (k=1, C3)
    orders an M-tile's spills after the previous tile's epilogue.

    ``e_ring`` >= 1: epilogue slots after the ring, chunk r_C in slot
    (rhat_C - 1) % e_ring, EPI->SPILL (k=e_ring) protecting them inside an
    M-tile and MMA->ACQL (k=1, C3) the ring across M-tiles (the next tile's
    loads reuse the slots).  ``e_ring`` = 0: chunk c of an M-tile in its own
    16 KiB of the ring; MMA->SPILL (k=0, C2 at M) starts the spills after the
    tile's last MFMAs and EPI->ACQL (k=1, C3) the next tile's loads after the
    epilogue read the chunks, so the MFMA engine spills a whole tile without
    waiting for the stores.

    ``linear``: MMA->LOAD is read with the linearized offset (an extension,
    not the paper's relation: k counts K iterations over all M-tiles of the
    workgroup, and the ring slot is (r_K - 1) % ring), which protects the
    ring across M-tiles by itself, so MMA->ACQL is dropped and the next
    tile's loads may start while the MFMAs of the previous tile run (with
    the epilogue in the ring, EPI->ACQL still holds them until the epilogue
    has read its chunks)."""
    k_dim, n_dim = (hidden, ffn) if phase == 1 else (ffn, hidden)
    ring = MOE_RINGS[bm, phase][0] if ring is None else ring
    e_ring = MOE_RINGS[bm, phase][1] if e_ring is None else e_ring
    b = ProgramBuilder("moe", n_engines=3, waves_per_engine=[2, 8, 2])
    with b.loop("M"):
        b.instr(0, OP_NOP, [0] * 8, name="ACQL")
        with b.loop("K"):
            b.instr(0, OP_MOE_LOAD, [phase, k_dim, n_dim, ring, bm, 0, 0, 0], name="LOAD")
            b.instr(1, OP_MOE_MMA, [0] * 8, name="MMA")
        b.instr(1, OP_NOP, [0] * 8, name="ACQE")
        with b.loop("C"):
            b.instr(1, OP_MOE_SPILL, [e_ring, 0, 0, 0, 0, 0, 0, 0], name="SPILL")
            b.instr(2, OP_MOE_EPI, [0] * 8, name="EPI")
    b.dep("LOAD", "MMA", 0)
    b.dep("MMA", "LOAD", ring, linear=linear)
    b.dep("SPILL", "EPI", 0)
    if e_ring == 0:
        # the M-tile's chunks in the ring: spills after the tile's last
        # MFMAs, the next tile's loads after the epilogue read the chunks
        b.dep("MMA", "SPILL", 0)
        b.dep("EPI", "ACQL", 1)
    else:
        b.dep("EPI", "SPILL", e_ring)
        if not linear:
            b.dep("MMA", "ACQL", 1)
    b.dep("EPI", "ACQE", 1)
    return b.build()


@dataclass
class MoeWork:
    work: np.ndarray      # int32 [n_wg, 4]: expert, first output column, first M-tile, M-tiles
    trips: TripTables     # per workgroup: [[1], [n_mt], [K / 32] * n_mt, [chunks] * n_mt]


def moe_worklist(counts, phase: int, hidden: int, ffn: int, mchunk: int = None, xcds: int = 8,
                 bm: int = MOE_BM) -> MoeWork:
    """Work items (expert, N-tile, run of at most ``mchunk`` M-tiles) in launch
    order.

    An expert's M-tiles are split into runs of nearly equal length.  The unit
    placed on an XCD is one (expert, N-tile) with all its runs: those
    workgroups stream the same weight rows in the same K order, so on one L2
    each weight chunk is fetched once for all runs.  Experts are taken
    largest first and each fills the least-loaded XCD up to an even share
    before spilling to the next, so an expert's token rows are shared by the
    N-tiles on the same XCD.  Workgroup w runs on XCD w % xcds; shorter XCD
    lists are padded with empty items (no M-tiles)."""
    k_dim, n_dim = (hidden, ffn) if phase == 1 else (ffn, hidden)
    mchunk = MOE_MCHUNKS[bm] if mchunk is None else mchunk
    bn = MOE_BN[phase]
    n_tiles = n_dim // bn
    counts = np.asarray(counts, dtype=np.int64)
    order = sorted(range(len(counts)), key=lambda e: (-int(counts[e]), e))
    mtiles = {e: -(-int(counts[e]) // bm) for e in order}
    share = sum(mtiles.values()) * n_tiles / xcds
    load = [0] * xcds
    lists = [[] for _ in range(xcds)]
    for e in order:
        mt = mtiles[e]
        if mt == 0:
            continue
        runs_n = -(-mt // mchunk)
        base, extra = divmod(mt, runs_n)
        runs, first = [], 0
        for r in range(runs_n):
            n_mt = base + (1 if r < extra else 0)
            runs.append((first, n_mt))
            first += n_mt
        t = 0
        while t < n_tiles:
            x = min(range(xcds), key=lambda i: (load[i], i))
            room = max(1, int((share - load[x]) // mt)) if load[x] < share else 1
            for tt in range(t, min(n_tiles, t + room)):
                for first, n_mt in runs:
                    lists[x].append((e, tt * bn, first, n_mt))
                load[x] += mt
            t += room
    depth = max((len(l) for l in lists), default=0)
    items = []
    for i in range(depth):
        for x in range(xcds):
            items.append(lists[x][i] if i < len(lists[x]) else (0, 0, 0, 0))
    work = np.array(items, dtype=np.int32).reshape(-1, 4)
    ksteps, chunks = k_dim // MOE_BK, moe_chunks(phase, bm)
    trips = TripTables([[np.array([1], np.int32), np.array([n_mt], np.int32),
                         np.full(n_mt, ksteps, np.int32), np.full(n_mt, chunks, np.int32)]
                        for _, _, _, n_mt in work])
    return MoeWork(work, trips)


# ---------------------------------------------------------------------------
# RMSNorm + FP8 quantization: a software-pipelined row loop
# ---------------------------------------------------------------------------
RMS_T, RMS_H = 32768, 8192


def rmsnorm_program(t: int = RMS_T, h: int = RMS_H, waves: int = 4, x_ring: int = 2, q_ring: int = 2,
                    eps: float = 1e-6) -> Program:
    """Load / vector / store engines over one row loop per workgroup, one
    row per iteration:

      R{ E0:LOAD X row -> xring[(rhat_R-1) % x_ring]
         E1:NORM xring -> codes + scale in qring[(rhat_R-1) % q_ring]
         E2:STORE qring -> Q, S }

    LOAD->NORM and NORM->STORE at offset 0 carry the data; NORM->LOAD at
    offset x_ring and STORE->NORM at offset q_ring keep a slot from being
    refilled before it is read (with two slots each: double buffering,
    offsets {0, 2}).  The vector engine's ``waves`` waves share each row
    (one column block each)."""
    b = ProgramBuilder("rmsnorm", n_engines=3, waves_per_engine=[1, waves, 1])
    with b.loop("R"):
        b.instr(0, OP_RMS_LOAD, [t, h, x_ring, 0, 0, 0, 0, 0], name="LOAD")
        b.instr(1, OP_RMS_NORM, [q_ring, f32_bits(eps), 0, 0, 0, 0, 0, 0], name="NORM")
        b.instr(2, OP_RMS_STORE, [0] * 8, name="STORE")
    b.dep("LOAD", "NORM", 0)
    b.dep("NORM", "LOAD", x_ring)
    b.dep("NORM", "STORE", 0)
    b.dep("STORE", "NORM", q_ring)
    return b.build()


def rmsnorm_worklist(t: int, n_wg: int):
    """Contiguous, balanced runs of rows per workgroup: (first row per
    workgroup int64 [n_wg], trip tables)."""
    start = (np.arange(n_wg + 1, dtype=np.int64) * t) // n_wg
    base = start[:-1].astype(np.int64)
    per = [[np.array([1], np.int32), np.array([int(start[w + 1] - start[w])], np.int32)] for w in range(n_wg)]
    return base, TripTables(per)


# ---------------------------------------------------------------------------
# AdamW over parameter chunks
# ---------------------------------------------------------------------------
ADAM_N = 1 << 20
ADAM_HP = dict(lr=1e-3, b1=0.9, b2=0.999, eps=1e-8, wd=0.01, t=10)


def adamw_program(n: int = ADAM_N, chunk: int = 1024, waves: int = 2, ring: int = 2, lr: float = 1e-3,
                  b1: float = 0.9, b2: float = 0.999, eps: float = 1e-8, wd: float = 0.01, t: int = 10) -> Program:
    """Load / vector / store engines over one loop of parameter chunks per
    workgroup, updating in place in the ring slot:

      C{ E0:LOAD p, g, m, v chunk -> ring[(rhat_C-1) % ring]
         E1:UPDATE AdamW on the slot (p, m, v rewritten)
         E2:STORE p, m, v -> HBM }

    LOAD->UPDATE and UPDATE->STORE at offset 0, STORE->LOAD at offset ring
    (with two slots: offsets {0, 2})."""
    b = ProgramBuilder("adamw", n_engines=3, waves_per_engine=[1, waves, 1])
    with b.loop("C"):
        b.instr(0, OP_ADAM_LOAD, [n, chunk, ring, 0, 0, 0, 0, 0], name="LOAD")
        b.instr(1, OP_ADAM_UPDATE, [f32_bits(lr), f32_bits(b1), f32_bits(b2), f32_bits(eps), f32_bits(wd), t, 0, 0],
                name="UPDATE")
        b.instr(2, OP_ADAM_STORE, [0] * 8, name="STORE")
    b.dep("LOAD", "UPDATE", 0)
    b.dep("UPDATE", "STORE", 0)
    b.dep("STORE", "LOAD", ring)
    return b.build()


def adamw_default_wg(n: int, chunk: int = 1024) -> int:
    """Workgroups of the benchmark launch shape: two chunks per workgroup,
    at most 1024 workgroups (512 for 2^20 parameters in chunks of 1024)."""
    n_chunks = -(-n // chunk)
    return max(1, min(1024, -(-n_chunks // 2)))


def adamw_worklist(n: int, chunk: int, n_wg: int):
    """Balanced contiguous runs of chunks per workgroup (the last chunk may
    be partial): (first chunk per workgroup int64 [n_wg], trip tables)."""
    n_chunks = -(-n // chunk)
    start = (np.arange(n_wg + 1, dtype=np.int64) * n_chunks) // n_wg
    per = [[np.array([1], np.int32), np.array([int(start[w + 1] - start[w])], np.int32)] for w in range(n_wg)]
    return start[:-1].astype(np.int64), TripTables(per)
