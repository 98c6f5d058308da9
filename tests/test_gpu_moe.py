"""GPU parity of the MoE grouped-GEMM family (load / MFMA / epilogue engines,
runtime M-tile loop per workgroup, two phases).

bf16 MFMA stages: |gpu - oracle| <= 2e-2 * max(|oracle|, rms(oracle)) per
element against the fp64 oracle (the GPU rounds h to bf16 between the two
phases, the oracle does not); thresholds bit-exact against the oracle's
brute force for every wave of every consumer engine; the barrier-free and
barrier modes produce bit-identical outputs."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import core, mathref  # noqa: E402
from paper_2608_13757_amd import (ALLOC_PER_INSTR, ALLOC_PER_LOOP, MODE_BARRIER, MODE_BARRIER_FREE,  # noqa: E402
                                  BfsError, Plan, bfs)
from tests.gpu_util import compare_wave_logs_with_oracle, log_records, trip_tensors  # noqa: E402
from workloads import moe_program, moe_worklist  # noqa: E402
from workloads.configs import MOE_BM, MOE_LINEAR, MOE_MCHUNKS  # noqa: E402
from workloads.tensors import bf16_to_f32, moe_inputs, moe_weights_all, to_bf16_bits  # noqa: E402

pytestmark = pytest.mark.gpu

MODES = [("barrier_free", MODE_BARRIER_FREE), ("barrier", MODE_BARRIER)]
RTOL = 2e-2


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bfs.lib()


def _say(*a):
    print(*a, flush=True, file=sys.stderr)


def _dev16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


class MoeRun:
    """Device copies of one MoE problem and the two launches."""

    def __init__(self, moe, mchunk=None, bm=MOE_BM):
        self.moe = moe
        wg, wu, wd = moe_weights_all(moe)
        self.wg, self.wu, self.wd = _dev16(wg), _dev16(wu), _dev16(wd)
        self.x = _dev16(moe.x)
        self.perm = torch.from_numpy(moe.perm.astype(np.int32)).cuda()
        self.eoff = torch.from_numpy(moe.expert_off.astype(np.int32)).cuda()
        T = len(moe.assign)
        self.h = torch.full((T, moe.ffn), -1, dtype=torch.int16, device="cuda")
        self.y = torch.full((T, moe.hidden), -1, dtype=torch.int16, device="cuda")
        self.set_mchunk(mchunk, bm)

    def set_mchunk(self, mchunk=None, bm=MOE_BM):
        """Work lists of ``bm``-token M-tiles with runs of at most ``mchunk``
        M-tiles per workgroup (the default for that tile height if None)."""
        self.mchunk, self.bm = (MOE_MCHUNKS[bm] if mchunk is None else mchunk), bm
        self.wl = {ph: moe_worklist(self.moe.counts, ph, self.moe.hidden, self.moe.ffn, mchunk=self.mchunk, bm=bm)
                   for ph in (1, 2)}
        self.dev_wl = {}
        for ph, wl in self.wl.items():
            trips, toff = trip_tensors(wl.trips)
            self.dev_wl[ph] = (torch.from_numpy(wl.work.reshape(-1)).cuda(), trips, toff, wl.trips.n_wg)

    def bufs(self, ph):
        work = self.dev_wl[ph][0]
        if ph == 1:
            return [work, self.perm, self.eoff, self.x, self.wg, self.wu, self.h]
        return [work, self.perm, self.eoff, self.h, self.wd, self.y]

    def run(self, mode, cap=0, alloc=ALLOC_PER_LOOP, linear=False, ring=None, e_ring=None):
        logs = {}
        for ph in (1, 2):
            plan = Plan(moe_program(ph, self.moe.hidden, self.moe.ffn, linear=linear, bm=self.bm, ring=ring,
                                    e_ring=e_ring), mode, alloc)
            work, trips, toff, n_wg = self.dev_wl[ph]
            log = None
            if cap:
                log = torch.zeros(plan.debug_log_words(n_wg, cap), dtype=torch.int32, device="cuda")
            plan.run(self.bufs(ph), trips, toff, n_wg, debug_log=log, debug_capacity=cap)
            plan.status()
            if cap:
                logs[ph] = (plan, log.cpu().numpy().view(np.uint32))
        h = bf16_to_f32(self.h.cpu().numpy().view(np.uint16))
        y = bf16_to_f32(self.y.cpu().numpy().view(np.uint16))
        return h, y, logs


def check_close(got, ref):
    ref = np.asarray(ref, np.float64)
    scale = np.maximum(np.abs(ref), np.sqrt(np.mean(ref ** 2)))
    err = np.abs(got.astype(np.float64) - ref) / scale
    assert np.isfinite(got).all()
    assert err.max() <= RTOL, (err.max(), np.unravel_index(err.argmax(), err.shape))
    return err.max()


# an empty expert, a one-token expert, ragged tiles, runs of M-tiles split
# over workgroups (mchunk 2)
SMALL_COUNTS = [300, 0, 129, 1, 530]
BMS = [128, 256]


@pytest.mark.parametrize("bm", BMS)
def test_moe_small_parity_and_thresholds(bm):
    moe = moe_inputs(seed=1, hidden=256, ffn=256, counts=SMALL_COUNTS)
    r = MoeRun(moe, mchunk=2, bm=bm)
    T = len(moe.assign)
    ref_y = mathref.moe_tokens(moe, range(T))
    grouped = moe.perm                                  # h rows are in expert-grouped order
    ref_h = mathref.moe_hidden(moe, grouped)
    outs = {}
    for name, mode in MODES:
        _say(f"[moe-small] bm={bm} mode={name}")
        h, y, logs = r.run(mode, cap=64)
        check_close(h, ref_h)
        check_close(y, ref_y)
        for ph in (1, 2):
            plan, logw = logs[ph]
            prog = moe_program(ph, moe.hidden, moe.ffn, bm=bm)
            wl = r.wl[ph]
            trips, off = wl.trips.flat()
            recs = {g: core.run(prog, trips, off[g], g).recs for g in range(wl.trips.n_wg)}
            lg = log_records(plan, logw, wl.trips.n_wg, 64, per_wave=True)
            assert compare_wave_logs_with_oracle(prog, plan, lg, recs, name) > 0
        outs[name] = y
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


@pytest.mark.parametrize("bm", BMS)
def test_moe_large_gate_values(bm):
    """x scaled by 256 (exact in bf16): gate and up pre-activations with a
    standard deviation near 80 reach SiLU's tails, where exp(-g) overflows to
    infinity for the most negative gates (SiLU(g) = -0) and SiLU(g) = g for
    the positive ones.  h and y against the oracle, both modes
    bit-identical."""
    moe = moe_inputs(seed=4, hidden=256, ffn=256, counts=SMALL_COUNTS)
    moe.x = to_bf16_bits(bf16_to_f32(moe.x) * 256.0)
    r = MoeRun(moe, mchunk=2, bm=bm)
    T = len(moe.assign)
    ref_y = mathref.moe_tokens(moe, range(T))
    ref_h = mathref.moe_hidden(moe, moe.perm)
    outs = {}
    for name, mode in MODES:
        _say(f"[moe-large] bm={bm} mode={name}")
        h, y, _ = r.run(mode)
        check_close(h, ref_h)
        check_close(y, ref_y)
        outs[name] = y
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


@pytest.mark.parametrize("bm", BMS)
def test_moe_linear_ring_parity_and_thresholds(bm):
    """MMA->LOAD read with the linearized offset (an extension) in place of
    the M-tile drain: outputs equal the oracle's and, bit for bit, the
    drained program's in both modes; every logged barrier-free threshold
    equals the brute force of the linearized relation (the paper's for the
    other dependencies), across M-tile boundaries (runs of 3 M-tiles)."""
    moe = moe_inputs(seed=2, hidden=256, ffn=256, counts=SMALL_COUNTS)
    r = MoeRun(moe, mchunk=3, bm=bm)
    T = len(moe.assign)
    ref_y = mathref.moe_tokens(moe, range(T))
    ref_h = mathref.moe_hidden(moe, moe.perm)
    _say("[moe-linear] drained program")
    h0, y0, _ = r.run(MODE_BARRIER_FREE)
    for name, mode in MODES:
        _say(f"[moe-linear] bm={bm} mode={name}")
        h, y, logs = r.run(mode, cap=64, linear=True)
        check_close(h, ref_h)
        check_close(y, ref_y)
        assert np.array_equal(h.view(np.uint32), h0.view(np.uint32))
        assert np.array_equal(y.view(np.uint32), y0.view(np.uint32))
        if name != "barrier_free":
            continue
        for ph in (1, 2):
            plan, logw = logs[ph]
            prog = moe_program(ph, moe.hidden, moe.ffn, linear=True, bm=bm)
            d_lin = [i for i, x in enumerate(prog.dep_linear) if x]
            wl = r.wl[ph]
            trips, off = wl.trips.flat()
            recs = {}
            for g in range(wl.trips.n_wg):
                res = core.run(prog, trips, off[g], g)
                rr = res.recs.copy()
                for d in d_lin:
                    rr[rr["dep"] == d] = core.linearized_records(prog, res, d)
                recs[g] = rr
            lg = log_records(plan, logw, wl.trips.n_wg, 64, per_wave=True)
            assert compare_wave_logs_with_oracle(prog, plan, lg, recs, name) > 0


@pytest.mark.parametrize("bm", BMS)
def test_moe_per_instr(bm):
    """One counter per producer instruction (Eq. 3): thresholds equal the
    Eq. 1 counts for every wave, values as with per-loop counters."""
    moe = moe_inputs(seed=3, hidden=256, ffn=256, counts=SMALL_COUNTS)
    r = MoeRun(moe, mchunk=2, bm=bm)
    _say(f"[moe-per-instr] bm={bm}")
    h, y, logs = r.run(MODE_BARRIER_FREE, cap=64, alloc=ALLOC_PER_INSTR)
    check_close(y, mathref.moe_tokens(moe, range(len(moe.assign))))
    for ph in (1, 2):
        plan, logw = logs[ph]
        prog = moe_program(ph, moe.hidden, moe.ffn, bm=bm)
        wl = r.wl[ph]
        trips, off = wl.trips.flat()
        recs = {g: core.run(prog, trips, off[g], g).recs for g in range(wl.trips.n_wg)}
        lg = log_records(plan, logw, wl.trips.n_wg, 64, per_wave=True)
        assert compare_wave_logs_with_oracle(prog, plan, lg, recs, "per_instr") > 0
    _, y2, _ = r.run(MODE_BARRIER_FREE)
    assert np.array_equal(y.view(np.uint32), y2.view(np.uint32))


@pytest.mark.parametrize("bm,layouts", [(128, [(5, 0), (5, 1), (5, 2)]), (256, [(4, 0), (4, 1), (3, 2)])])
def test_moe_epilogue_layouts(bm, layouts):
    """Both epilogue layouts in both phases: (ring, epilogue slots) with the
    chunks in the K ring (0: MMA->SPILL and EPI->ACQL) or in 1 or 2 slots
    after it (EPI->SPILL and MMA->ACQL); outputs equal the oracle's and,
    bit for bit, each other in both modes, and every logged threshold equals
    the oracle's.  A layout beyond 160 KiB of LDS is refused."""
    moe = moe_inputs(seed=4, hidden=256, ffn=256, counts=SMALL_COUNTS)
    r = MoeRun(moe, mchunk=2, bm=bm)
    ref_y = mathref.moe_tokens(moe, range(len(moe.assign)))
    first = None
    for ring, e_ring in layouts:
        for name, mode in MODES:
            _say(f"[moe-epilogue] bm={bm} ring={ring} e_ring={e_ring} mode={name}")
            h, y, logs = r.run(mode, cap=64, ring=ring, e_ring=e_ring)
            check_close(y, ref_y)
            for ph in (1, 2):
                plan, logw = logs[ph]
                prog = moe_program(ph, moe.hidden, moe.ffn, bm=bm, ring=ring, e_ring=e_ring)
                wl = r.wl[ph]
                trips, off = wl.trips.flat()
                recs = {g: core.run(prog, trips, off[g], g).recs for g in range(wl.trips.n_wg)}
                lg = log_records(plan, logw, wl.trips.n_wg, 64, per_wave=True)
                assert compare_wave_logs_with_oracle(prog, plan, lg, recs, name) > 0
            if first is None:
                first = (h, y)
            assert np.array_equal(h.view(np.uint32), first[0].view(np.uint32))
            assert np.array_equal(y.view(np.uint32), first[1].view(np.uint32))
    if bm == 256:
        with pytest.raises(BfsError) as e:
            r.run(MODE_BARRIER_FREE, ring=4, e_ring=2)
        assert e.value.status == bfs.E_RESOURCE


@pytest.fixture(scope="module")
def full_moe():
    """The benchmark problem (32768 tokens, 64 Zipf(1.1) experts, hidden
    4096, ffn 1408, seed 0) on the device, and the oracle's y rows of
    sampled tokens and h rows of sampled expert-grouped positions."""
    _say("[moe-full] generating")
    moe = moe_inputs(seed=0)
    r = MoeRun(moe)
    order = np.argsort(-moe.counts)
    experts = list(order[:3]) + list(order[30:32]) + list(order[-3:])   # largest, middle, smallest
    rng = np.random.default_rng(5)
    tokens, rows = [], []
    for e in experts:
        lo, hi = int(moe.expert_off[e]), int(moe.expert_off[e + 1])
        group = moe.perm[lo:hi]
        tokens += [int(group[0]), int(group[-1])] + [int(t) for t in rng.choice(group, 6)]
        # h rows are in expert-grouped order: the first and last row of the
        # expert, the first row of its last (ragged) M-tile at both tile
        # heights, and random ones
        rows += [lo, hi - 1, lo + (hi - 1 - lo) // 128 * 128, lo + (hi - 1 - lo) // 256 * 256]
        rows += [int(i) for i in rng.integers(lo, hi, 4)]
    weights = {}
    ref_y = mathref.moe_tokens(moe, tokens, weights)
    ref_h = mathref.moe_hidden(moe, [int(moe.perm[i]) for i in rows], weights)
    return r, tokens, ref_y, rows, ref_h


OTHER_BM = 256 if MOE_BM == 128 else 128


@pytest.mark.parametrize("mchunk,linear,bm", [(None, MOE_LINEAR, MOE_BM), (None, not MOE_LINEAR, MOE_BM),
                                              (8, MOE_LINEAR, MOE_BM), (None, MOE_LINEAR, OTHER_BM)],
                         ids=["bench", "bench_other_form", "m8", "other_bm"])
def test_moe_full_size_sampled(full_moe, mchunk, linear, bm):
    """The benchmark shape and launch (the default M-tile height and runs,
    the paper's ACQL drain, as timed), then the linearized ring, runs of
    eight M-tiles, and the other M-tile height; sampled y tokens and h rows
    one by one; both modes bit-identical."""
    r, tokens, ref_y, rows, ref_h = full_moe
    r.set_mchunk(mchunk, bm)
    outs = {}
    for name, mode in MODES:
        _say(f"[moe-full] bm={bm} mchunk={r.mchunk} linear={linear} mode={name}")
        r.h.fill_(-1)
        r.y.fill_(-1)
        h, y, _ = r.run(mode, linear=linear)
        check_close(y[tokens], ref_y)
        check_close(h[rows], ref_h)
        outs[name] = (h, y)
    for a, b in zip(outs["barrier_free"], outs["barrier"]):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_moe_rejects_missing_dependency():
    prog = moe_program(1, 256, 256)
    prog.deps = [d for d in prog.deps if prog.instrs[d[1]].name != "ACQL"]
    plan = Plan(prog)
    t = torch.zeros(16, dtype=torch.int32, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([t] * 7, t, t, 1)
    assert e.value.status == bfs.E_UNSUPPORTED


def test_moe_watchdog():
    moe = moe_inputs(seed=3, hidden=256, ffn=256, counts=[200, 50])
    r = MoeRun(moe)
    plan = Plan(moe_program(1, moe.hidden, moe.ffn))
    work, trips, toff, n_wg = r.dev_wl[1]
    _say("[moe-watchdog]")
    plan.run(r.bufs(1), trips, toff, n_wg, watchdog_polls=2000, fault_dep=0, fault_delta=1 << 20)
    with pytest.raises(BfsError) as e:
        plan.status()
    assert e.value.status == bfs.E_DEADLOCK
    plan.run(r.bufs(1), trips, toff, n_wg)
    plan.status()
