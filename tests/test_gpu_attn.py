"""GPU parity of the variable-length attention family (K load / QK^T MFMA /
online softmax / PV MFMA / V load engines).

bf16 MFMA stages: |gpu - oracle| <= 2e-2 * max(|oracle|, rms(oracle)) per
element against the fp64 oracle; thresholds bit-exact against the oracle's
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
from workloads import attn_program, attn_worklist  # noqa: E402
from workloads.configs import ATTN_LINEAR, ATTN_NK, ATTN_NV, ATTN_WG  # noqa: E402
from workloads.tensors import attn_inputs, bf16_to_f32, to_bf16_bits  # noqa: E402

pytestmark = pytest.mark.gpu

MODES = [("barrier_free", MODE_BARRIER_FREE), ("barrier", MODE_BARRIER)]
RTOL = 2e-2
SCALE = 1.0 / np.sqrt(128.0)


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bfs.lib()


def _say(*a):
    print(*a, flush=True, file=sys.stderr)


def _dev16(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()


def run_attn(ai, heads, mode, cap=0, nk=ATTN_NK, nv=ATTN_NV, alloc=ALLOC_PER_LOOP, n_wg=ATTN_WG, linear=ATTN_LINEAR):
    prog = attn_program(heads, nk=nk, nv=nv, linear=linear)
    plan = Plan(prog, mode, alloc)
    wl = attn_worklist(ai.lengths, heads, n_wg=n_wg)
    trips, toff = trip_tensors(wl.trips)
    work = torch.from_numpy(wl.work.reshape(-1)).cuda()
    q, k, v = _dev16(ai.q), _dev16(ai.k), _dev16(ai.v)
    o = torch.full(ai.q.shape, -1, dtype=torch.int16, device="cuda")
    n_wg = wl.trips.n_wg
    log = None
    if cap:
        log = torch.zeros(plan.debug_log_words(n_wg, cap), dtype=torch.int32, device="cuda")
    plan.run([work, q, k, v, o], trips, toff, n_wg, debug_log=log, debug_capacity=cap)
    plan.status()
    out = bf16_to_f32(o.cpu().numpy().view(np.uint16))
    return prog, plan, wl, out, (log.cpu().numpy().view(np.uint32) if cap else None)


def oracle_recs(prog, wl):
    """The oracle's records per workgroup; the ring and S/P reuse
    dependencies (read with the linearized offset) take the brute force of
    that relation."""
    trips, off = wl.trips.flat()
    out = {}
    for g in range(wl.trips.n_wg):
        res = core.run(prog, trips, off[g], g)
        rr = res.recs.copy()
        for d, lin in enumerate(prog.dep_linear):
            if lin:
                rr[rr["dep"] == d] = core.linearized_records(prog, res, d)
        out[g] = rr
    return out


def check_close(got, ref):
    ref = np.asarray(ref, np.float64)
    scale = np.maximum(np.abs(ref), np.sqrt(np.mean(ref ** 2)))
    err = np.abs(got.astype(np.float64) - ref) / scale
    assert np.isfinite(got).all()
    assert err.max() <= RTOL, (err.max(), np.unravel_index(err.argmax(), err.shape))
    return err.max()


# lengths: one key, exactly one block, a ragged block, two query tiles with
# a one-row tail, several blocks with a ragged last block
SMALL = [1, 64, 100, 129, 300]


@pytest.mark.parametrize("rings,n_wg", [((3, 2), 3), ((2, 2), 3), ((2, 3), 3), ((3, 2), 64)])
def test_attn_small_parity_and_thresholds(rings, n_wg):
    """The linearized form: three workgroups run all 16 tiles (several tiles
    each, so the rings, S/P slots and row sums cross tile boundaries); 64
    workgroups leave most with one tile or none."""
    nk, nv = rings
    heads = 2
    ai = attn_inputs(seed=1, heads=heads, lengths=SMALL)
    ref = mathref.attention(ai.q, ai.k, ai.v, ai.cu_seqlens, SCALE)
    outs = {}
    for name, mode in MODES:
        _say(f"[attn-small] rings={rings} n_wg={n_wg} mode={name}")
        prog, plan, wl, out, logw = run_attn(ai, heads, mode, cap=256, nk=nk, nv=nv, n_wg=n_wg, linear=True)
        check_close(out, ref)
        recs = oracle_recs(prog, wl)
        logs = log_records(plan, logw, wl.trips.n_wg, 256, per_wave=True)
        assert compare_wave_logs_with_oracle(prog, plan, logs, recs, name) > 0
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


@pytest.mark.parametrize("rings,n_wg", [((2, 3), 3), ((3, 2), 3), ((2, 2), 64)])
def test_attn_acquire_form_parity_and_thresholds(rings, n_wg):
    """The paper's relation only: per-trip reuse dependencies and acquire
    instructions at each tile (C3 drains of the previous tile's QK, PV and
    PREAD).  Values against the oracle, every wave's thresholds equal to the
    brute force of Eq. 1, both modes bit-identical, and equal to the
    linearized form's output."""
    nk, nv = rings
    heads = 2
    ai = attn_inputs(seed=5, heads=heads, lengths=SMALL)
    ref = mathref.attention(ai.q, ai.k, ai.v, ai.cu_seqlens, SCALE)
    outs = {}
    for name, mode in MODES:
        _say(f"[attn-acq] rings={rings} n_wg={n_wg} mode={name}")
        prog, plan, wl, out, logw = run_attn(ai, heads, mode, cap=256, nk=nk, nv=nv, n_wg=n_wg, linear=False)
        check_close(out, ref)
        recs = oracle_recs(prog, wl)
        logs = log_records(plan, logw, wl.trips.n_wg, 256, per_wave=True)
        assert compare_wave_logs_with_oracle(prog, plan, logs, recs, name) > 0
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))
    _, _, _, lin, _ = run_attn(ai, heads, MODE_BARRIER_FREE, nk=nk, nv=nv, n_wg=n_wg, linear=True)
    assert np.array_equal(outs["barrier_free"].view(np.uint32), lin.view(np.uint32))


def test_attn_tiles_beyond_staged_descriptors():
    """One workgroup runs 700 tiles (700 sequences of 1 to 128 keys, one
    head): the kernel stages the first tile descriptors in the LDS left over
    by the rings (614 of them at the benchmark's rings) and reads the rest
    from memory.  Values against the oracle, both modes bit-identical."""
    heads = 1
    lengths = np.random.default_rng(7).integers(1, 129, 700)
    ai = attn_inputs(seed=7, heads=heads, lengths=lengths)
    ref = mathref.attention(ai.q, ai.k, ai.v, ai.cu_seqlens, SCALE)
    outs = {}
    for name, mode in MODES:
        _say(f"[attn-many-tiles] mode={name}")
        _, _, wl, out, _ = run_attn(ai, heads, mode, n_wg=1)
        assert len(wl.trips.per_wg[0][2]) == 700
        check_close(out, ref)
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


def test_attn_per_instr():
    """One counter per producer instruction (Eq. 3): thresholds equal the
    Eq. 1 counts for every wave, values as with per-loop counters."""
    heads = 2
    ai = attn_inputs(seed=4, heads=heads, lengths=SMALL)
    _say("[attn-per-instr]")
    prog, plan, wl, out, logw = run_attn(ai, heads, MODE_BARRIER_FREE, cap=256, alloc=ALLOC_PER_INSTR, n_wg=3)
    check_close(out, mathref.attention(ai.q, ai.k, ai.v, ai.cu_seqlens, SCALE))
    recs = oracle_recs(prog, wl)
    logs = log_records(plan, logw, wl.trips.n_wg, 256, per_wave=True)
    assert compare_wave_logs_with_oracle(prog, plan, logs, recs, "per_instr") > 0
    _, _, _, out2, _ = run_attn(ai, heads, MODE_BARRIER_FREE, n_wg=3)
    assert np.array_equal(out.view(np.uint32), out2.view(np.uint32))


def test_attn_special_cases():
    """Constant V rows give O = that row; a one-token sequence returns its V."""
    heads = 2
    ai = attn_inputs(seed=2, heads=heads, lengths=[1, 200])
    const = ai.v[1].copy()                          # token 1 is the first of sequence 1
    ai.v[1:] = const[None]
    _say("[attn-special]")
    _, _, _, out, _ = run_attn(ai, heads, MODE_BARRIER_FREE)
    check_close(out[0], bf16_to_f32(ai.v[0]))
    check_close(out[1:], np.broadcast_to(bf16_to_f32(const), out[1:].shape))


def test_attn_peaked_and_flat_softmax():
    """Large and vanishing logits.  Q scaled by 16 (an exact power of two in
    bf16): scores with a standard deviation near 180 make the softmax nearly
    one-hot and move the running maximum by large steps between KV blocks,
    so the rescale factor underflows to 0 for some rows.  A sequence with
    Q = 0 weights its keys equally: every block after the first keeps the
    running maximum (a rescale by exactly 1, which the kernel skips) and O
    is the mean of V.  Values against the oracle, both modes bit-identical."""
    heads = 2
    ai = attn_inputs(seed=9, heads=heads, lengths=[300, 1000, 129, 700])
    q = bf16_to_f32(ai.q) * 16.0
    s3 = int(ai.cu_seqlens[3])
    q[s3:] = 0.0
    ai.q = to_bf16_bits(q)
    ref = np.asarray(mathref.attention(ai.q, ai.k, ai.v, ai.cu_seqlens, SCALE), np.float64)
    mean_v = bf16_to_f32(ai.v[s3:]).astype(np.float64).mean(axis=0)
    assert np.allclose(ref[s3:], mean_v[None], rtol=1e-9, atol=1e-12)
    outs = {}
    for name, mode in MODES:
        _say(f"[attn-peaked-flat] mode={name}")
        _, _, _, out, _ = run_attn(ai, heads, mode, n_wg=8)
        check_close(out, ref)
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


@pytest.fixture(scope="module")
def full_attn():
    """The benchmark inputs (32 sequences of U[128, 4096] tokens, 16 heads,
    seed 0) and the oracle's rows at sampled (sequence, head, row) items."""
    heads = 16
    _say("[attn-full] generating")
    ai = attn_inputs(seed=0, heads=heads)
    rng = np.random.default_rng(11)
    items = []
    for _ in range(200):
        b = int(rng.integers(0, len(ai.lengths)))
        items.append((b, int(rng.integers(0, heads)), int(rng.integers(0, ai.lengths[b]))))
    for b in range(len(ai.lengths)):                # first and last row of every sequence
        L = int(ai.lengths[b])
        items += [(b, b % heads, 0), (b, (b + 7) % heads, L - 1), (b, (b + 3) % heads, (L - 1) // 128 * 128)]
    ref = mathref.attention_rows(ai.q, ai.k, ai.v, ai.cu_seqlens, SCALE, items)
    return heads, ai, items, ref


@pytest.mark.parametrize("rings,linear", [((ATTN_NK, ATTN_NV), ATTN_LINEAR), ((ATTN_NK, ATTN_NV), not ATTN_LINEAR),
                                         ((3, 2), ATTN_LINEAR)], ids=["bench", "bench_other_form", "k3v2"])
def test_attn_full_size_sampled(full_attn, rings, linear):
    """The benchmark shape and launch (256 persistent workgroups, the
    benchmark's K and V ring depths and its acquire form; then the
    linearized form and the other ring layout), checked on sampled rows one
    by one; both modes bit-identical."""
    heads, ai, items, ref = full_attn
    nk, nv = rings
    outs = {}
    for name, mode in MODES:
        _say(f"[attn-full] rings={rings} linear={linear} mode={name}")
        _, _, wl, out, _ = run_attn(ai, heads, mode, nk=nk, nv=nv, linear=linear)
        assert wl.trips.n_wg == ATTN_WG
        got = np.array([out[ai.cu_seqlens[b] + i, h] for b, h, i in items])
        check_close(got, ref)
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


def test_attn_rejects_paper_relation_for_ring_reuse():
    """The kernel indexes the rings and S/P slots by r_KV over all tiles:
    a program whose reuse dependencies use the paper's per-trip relation
    would let a tile's first loads overwrite slots the previous tile still
    reads unless acquires drain them, so the launcher refuses it without
    the acquires (and refuses the acquire form with a drain missing)."""
    prog = attn_program(2, linear=True)
    prog.dep_linear = [0] * len(prog.deps)
    plan = Plan(prog)
    t = torch.zeros(16, dtype=torch.int32, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([t, t, t, t, t], t, t, 1)
    assert e.value.status == bfs.E_UNSUPPORTED
    prog = attn_program(2, linear=False)
    keep = [i for i, d in enumerate(prog.deps) if prog.instrs[d[1]].name != "ACQV"]
    prog.deps = [prog.deps[i] for i in keep]
    prog.dep_linear = [prog.dep_linear[i] for i in keep]
    plan = Plan(prog)
    t = torch.zeros(16, dtype=torch.int32, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([t, t, t, t, t], t, t, 1)
    assert e.value.status == bfs.E_UNSUPPORTED


def test_attn_rejects_missing_dependency():
    prog = attn_program(2)
    keep = [i for i, d in enumerate(prog.deps)
            if not (prog.instrs[d[0]].name == "PREAD" and prog.instrs[d[1]].name == "QK")]
    prog.deps = [prog.deps[i] for i in keep]
    prog.dep_linear = [prog.dep_linear[i] for i in keep]
    plan = Plan(prog)
    t = torch.zeros(16, dtype=torch.int32, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([t, t, t, t, t], t, t, 1)
    assert e.value.status == bfs.E_UNSUPPORTED


def test_attn_watchdog():
    heads = 1
    ai = attn_inputs(seed=3, heads=heads, lengths=[300])
    prog = attn_program(heads)
    plan = Plan(prog)
    wl = attn_worklist(ai.lengths, heads)
    trips, toff = trip_tensors(wl.trips)
    work = torch.from_numpy(wl.work.reshape(-1)).cuda()
    q, k, v = _dev16(ai.q), _dev16(ai.k), _dev16(ai.v)
    o = torch.zeros(ai.q.shape, dtype=torch.int16, device="cuda")
    _say("[attn-watchdog]")
    plan.run([work, q, k, v, o], trips, toff, wl.trips.n_wg, watchdog_polls=2000, fault_dep=2, fault_delta=1 << 20)
    with pytest.raises(BfsError) as e:
        plan.status()
    assert e.value.status == bfs.E_DEADLOCK
    plan.run([work, q, k, v, o], trips, toff, wl.trips.n_wg)
    plan.status()


def test_attn_rejects_trip_beyond_sequence():
    """A KV trip count longer than the sequence's blocks is clamped on the
    device and reported by bfs_run_status as an invalid input."""
    heads = 1
    ai = attn_inputs(seed=3, heads=heads, lengths=[100])
    prog = attn_program(heads)
    plan = Plan(prog)
    wl = attn_worklist(ai.lengths, heads)
    wl.trips.per_wg[0][2][0] += 1            # one KV block too many
    trips, toff = trip_tensors(wl.trips)
    work = torch.from_numpy(wl.work.reshape(-1)).cuda()
    q, k, v = _dev16(ai.q), _dev16(ai.k), _dev16(ai.v)
    o = torch.zeros(ai.q.shape, dtype=torch.int16, device="cuda")
    _say("[attn-bad-trip]")
    plan.run([work, q, k, v, o], trips, toff, wl.trips.n_wg)
    with pytest.raises(BfsError) as e:
        plan.status()
    assert e.value.status == bfs.E_INVALID
