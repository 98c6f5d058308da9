"""GPU parity of the GEMM + bias + GELU family (load / MFMA / epilogue engines).

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
from workloads import gemm_program, gemm_program_k_unrolled, gemm_trips, gemm_trips_k_unrolled  # noqa: E402
from workloads.tensors import bf16_to_f32, gemm_inputs  # noqa: E402

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


def _bits_to_dev(bits):
    return torch.from_numpy(bits.view(np.int16)).cuda()


def run_gemm(gi, m, n, k, mode, cap=0, alloc=ALLOC_PER_LOOP, e_ring=None):
    prog = gemm_program(m, n, k) if e_ring is None else gemm_program(m, n, k, e_ring=e_ring)
    plan = Plan(prog, mode, alloc)
    tt = gemm_trips(m, n, k)
    trips, toff = trip_tensors(tt)
    a, bt = _bits_to_dev(gi.a), _bits_to_dev(gi.bt)
    bias = torch.from_numpy(gi.bias).cuda()
    c = torch.full((m * n,), -1, dtype=torch.int16, device="cuda")
    log = None
    if cap:
        log = torch.zeros(plan.debug_log_words(tt.n_wg, cap), dtype=torch.int32, device="cuda")
    plan.run([a, bt, bias, c], trips, toff, tt.n_wg, debug_log=log, debug_capacity=cap)
    plan.status()
    out = bf16_to_f32(c.cpu().numpy().view(np.uint16)).reshape(m, n)
    return prog, plan, tt, out, (log.cpu().numpy().view(np.uint32) if cap else None)


def check_close(got, ref):
    ref = np.asarray(ref, np.float64)
    scale = np.maximum(np.abs(ref), np.sqrt(np.mean(ref ** 2)))
    err = np.abs(got.astype(np.float64) - ref) / scale
    assert np.isfinite(got).all()
    assert err.max() <= RTOL, (err.max(), np.unravel_index(err.argmax(), err.shape))
    return err.max()


@pytest.mark.parametrize("shape", [(512, 512, 256), (256, 768, 96)])
def test_gemm_k_unroll(shape):
    """K-loop bodies unrolled 2, 4 and 8 times (a remainder of single steps
    when the trip is not a multiple): bit-identical to the single bodies, in
    both modes."""
    m, n, k = shape
    gi = gemm_inputs(seed=3, m=m, n=n, k=k)
    prog = gemm_program(m, n, k)
    tt = gemm_trips(m, n, k)
    trips, toff = trip_tensors(tt)
    a, bt = _bits_to_dev(gi.a), _bits_to_dev(gi.bt)
    bias = torch.from_numpy(gi.bias).cuda()
    for name, mode in MODES:
        plan = Plan(prog, mode)
        outs = {}
        for u in (1, 2, 4, 8):
            _say(f"[gemm-unroll] {shape} mode={name} k_unroll={u}")
            c = torch.full((m * n,), -1, dtype=torch.int16, device="cuda")
            plan.run([a, bt, bias, c], trips, toff, tt.n_wg, k_unroll=u)
            plan.status()
            outs[u] = c.cpu().numpy()
        for u in (2, 4, 8):
            assert np.array_equal(outs[u], outs[1]), (name, u)
    check_close(bf16_to_f32(outs[1].view(np.uint16)).reshape(m, n), mathref.gemm_bias_gelu(gi.a, gi.bt, gi.bias))


@pytest.mark.parametrize("u", [2, 4, 8])
def test_gemm_k_unroll_thresholds(u):
    """The unrolled K bodies' waits, logged from the same unrolled code that
    uninstrumented launches time: every logged threshold equals the oracle's
    for every wave, in both modes (K trips 8: a multiple of every factor;
    3: all remainder for u >= 4)."""
    for m, n, k in ((512, 512, 256), (256, 768, 96)):
        gi = gemm_inputs(seed=5, m=m, n=n, k=k)
        prog = gemm_program(m, n, k)
        tt = gemm_trips(m, n, k)
        trips, toff = trip_tensors(tt)
        a, bt = _bits_to_dev(gi.a), _bits_to_dev(gi.bt)
        bias = torch.from_numpy(gi.bias).cuda()
        t_np, off = tt.flat()
        recs = {g: core.run(prog, t_np, off[g], g).recs for g in range(tt.n_wg)}
        outs = {}
        for name, mode in MODES:
            _say(f"[gemm-unroll-log] {(m, n, k)} u={u} mode={name}")
            plan = Plan(prog, mode)
            cap = 512
            log = torch.zeros(plan.debug_log_words(tt.n_wg, cap), dtype=torch.int32, device="cuda")
            c = torch.full((m * n,), -1, dtype=torch.int16, device="cuda")
            plan.run([a, bt, bias, c], trips, toff, tt.n_wg, debug_log=log, debug_capacity=cap, k_unroll=u)
            plan.status()
            logs = log_records(plan, log.cpu().numpy().view(np.uint32), tt.n_wg, cap, per_wave=True)
            assert compare_wave_logs_with_oracle(prog, plan, logs, recs, name) > 0
            outs[name] = c.cpu().numpy()
        assert np.array_equal(outs["barrier_free"], outs["barrier"])


@pytest.mark.parametrize("shape", [(512, 512, 256), (256, 768, 96), (512, 256, 4096)])
def test_gemm_k_unrolled_program(shape):
    """The K-unrolled program (K loop removed, the steps listed at the top
    level, every K-phase wait a static immediate): outputs bit-identical to
    the looped program's in both modes, every logged threshold equal to the
    oracle's for every wave."""
    m, n, k = shape
    gi = gemm_inputs(seed=6, m=m, n=n, k=k)
    a, bt = _bits_to_dev(gi.a), _bits_to_dev(gi.bt)
    bias = torch.from_numpy(gi.bias).cuda()
    prog = gemm_program_k_unrolled(m, n, k)
    tt = gemm_trips_k_unrolled(m, n)
    trips, toff = trip_tensors(tt)
    t_np, off = tt.flat()
    recs = {g: core.run(prog, t_np, off[g], g).recs for g in range(0, tt.n_wg, max(1, tt.n_wg // 3))}
    _, _, _, ref, _ = run_gemm(gi, m, n, k, MODE_BARRIER_FREE)
    for name, mode in MODES:
        _say(f"[gemm-k-unrolled] {shape} mode={name}")
        plan = Plan(prog, mode)
        cap = 512
        log = torch.zeros(plan.debug_log_words(tt.n_wg, cap), dtype=torch.int32, device="cuda")
        c = torch.full((m * n,), -1, dtype=torch.int16, device="cuda")
        plan.run([a, bt, bias, c], trips, toff, tt.n_wg, debug_log=log, debug_capacity=cap)
        plan.status()
        logs = log_records(plan, log.cpu().numpy().view(np.uint32), tt.n_wg, cap, per_wave=True)
        assert compare_wave_logs_with_oracle(prog, plan, logs, recs, name) > 0
        out = bf16_to_f32(c.cpu().numpy().view(np.uint16)).reshape(m, n)
        assert np.array_equal(out.view(np.uint32), ref.view(np.uint32))
        c.fill_(-1)
        plan.run([a, bt, bias, c], trips, toff, tt.n_wg)
        plan.status()
        assert np.array_equal(bf16_to_f32(c.cpu().numpy().view(np.uint16)).reshape(m, n).view(np.uint32),
                              ref.view(np.uint32))
    if k <= 256:
        check_close(ref, mathref.gemm_bias_gelu(gi.a, gi.bt, gi.bias))


def test_gemm_k_unrolled_rejects_other_steps():
    m, n, k = 256, 256, 64                     # 2 steps: no kernel built for it
    plan = Plan(gemm_program_k_unrolled(m, n, k))
    tt = gemm_trips_k_unrolled(m, n)
    trips, toff = trip_tensors(tt)
    t = torch.zeros(m * k, dtype=torch.int16, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([t, t, torch.zeros(n, device="cuda"), t], trips, toff, tt.n_wg)
    assert e.value.status == bfs.E_UNSUPPORTED


def test_gemm_k_unroll_rejects_other_factors():
    m, n, k = 256, 256, 64
    prog = gemm_program(m, n, k)
    plan = Plan(prog)
    tt = gemm_trips(m, n, k)
    trips, toff = trip_tensors(tt)
    t = torch.zeros(m * k, dtype=torch.int16, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([t, t, torch.zeros(n, device="cuda"), t], trips, toff, tt.n_wg, k_unroll=3)
    assert e.value.status == bfs.E_INVALID


def test_gemm_per_instr():
    """One counter per producer instruction (Eq. 3): thresholds equal the
    Eq. 1 counts for every wave, values as with per-loop counters."""
    m, n, k = 512, 512, 256
    gi = gemm_inputs(seed=2, m=m, n=n, k=k)
    _say("[gemm-per-instr]")
    prog, plan, tt, out, logw = run_gemm(gi, m, n, k, MODE_BARRIER_FREE, cap=512, alloc=ALLOC_PER_INSTR)
    check_close(out, mathref.gemm_bias_gelu(gi.a, gi.bt, gi.bias))
    trips, off = tt.flat()
    recs = {g: core.run(prog, trips, off[g], g).recs for g in range(tt.n_wg)}
    logs = log_records(plan, logw, tt.n_wg, 512, per_wave=True)
    assert compare_wave_logs_with_oracle(prog, plan, logs, recs, "per_instr") > 0
    _, _, _, out2, _ = run_gemm(gi, m, n, k, MODE_BARRIER_FREE)
    assert np.array_equal(out.view(np.uint32), out2.view(np.uint32))


@pytest.mark.parametrize("shape", [(512, 512, 256), (256, 768, 96)])
def test_gemm_small_parity_and_thresholds(shape):
    m, n, k = shape
    gi = gemm_inputs(seed=1, m=m, n=n, k=k)
    ref = mathref.gemm_bias_gelu(gi.a, gi.bt, gi.bias)
    outs = {}
    for name, mode in MODES:
        _say(f"[gemm-small] {shape} mode={name}")
        prog, plan, tt, out, logw = run_gemm(gi, m, n, k, mode, cap=512)
        check_close(out, ref)
        trips, off = tt.flat()
        recs = {g: core.run(prog, trips, off[g], g).recs for g in range(tt.n_wg)}
        logs = log_records(plan, logw, tt.n_wg, 512, per_wave=True)
        assert compare_wave_logs_with_oracle(prog, plan, logs, recs, name) > 0
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


def test_gemm_epilogue_rings():
    """Epilogue rings of 1, 2, 4 and 8 slots in the idle K ring (EPI->SPILL
    at offset = slots): every logged threshold equals the oracle's in both
    modes, outputs bit-identical across ring sizes and modes; sizes that are
    not a power of two, or larger than 8, are refused."""
    m, n, k = 512, 512, 256
    gi = gemm_inputs(seed=4, m=m, n=n, k=k)
    ref = mathref.gemm_bias_gelu(gi.a, gi.bt, gi.bias)
    outs = {}
    for e_ring in (1, 2, 4, 8):
        for name, mode in MODES:
            _say(f"[gemm-epilogue] e_ring={e_ring} mode={name}")
            prog, plan, tt, out, logw = run_gemm(gi, m, n, k, mode, cap=512, e_ring=e_ring)
            check_close(out, ref)
            trips, off = tt.flat()
            recs = {g: core.run(prog, trips, off[g], g).recs for g in range(tt.n_wg)}
            logs = log_records(plan, logw, tt.n_wg, 512, per_wave=True)
            assert compare_wave_logs_with_oracle(prog, plan, logs, recs, name) > 0
            outs[(e_ring, name)] = out
    first = next(iter(outs.values()))
    for key, out in outs.items():
        assert np.array_equal(out.view(np.uint32), first.view(np.uint32)), key
    for bad in (3, 16):
        with pytest.raises(BfsError) as e:
            run_gemm(gi, m, n, k, MODE_BARRIER_FREE, e_ring=bad)
        assert e.value.status == bfs.E_UNSUPPORTED


def test_gemm_special_cases():
    """B = I gives GELU(A + bias); A = 0 gives GELU(bias) in every row."""
    m, n, k = 256, 256, 256
    gi = gemm_inputs(seed=2, m=m, n=n, k=k)
    from workloads.tensors import to_bf16_bits
    gi.bt = to_bf16_bits(np.eye(n, k, dtype=np.float32))
    _say("[gemm-identity]")
    _, _, _, out, _ = run_gemm(gi, m, n, k, MODE_BARRIER_FREE)
    a = bf16_to_f32(gi.a).astype(np.float64)
    check_close(out, mathref.gelu(a + gi.bias[None, :].astype(np.float64)))
    gi.a = np.zeros_like(gi.a)
    _, _, _, out, _ = run_gemm(gi, m, n, k, MODE_BARRIER_FREE)
    check_close(out, np.broadcast_to(mathref.gelu(gi.bias.astype(np.float64)), (m, n)))


def test_gemm_gelu_range():
    """A = 0, so every row of C is GELU(bias) as the epilogue evaluates it:
    bias values from -64 to 64 (one per column) cover GELU's saturated tails
    and its curved middle.  Each element is within the bf16 output rounding
    (2^-8 relative) plus the erf approximation's error (1.5e-7 absolute in
    erf, and the fp32 cancellation in 1 + erf at negative arguments, both
    scaled by |x| / 2) of the exact-erf oracle; both modes bit-identical."""
    m, n, k = 256, 512, 64
    gi = gemm_inputs(seed=3, m=m, n=n, k=k)
    gi.a = np.zeros_like(gi.a)
    gi.bias = np.linspace(-64.0, 64.0, n).astype(np.float32)
    x = gi.bias.astype(np.float64)
    ref = mathref.gelu(x)
    bound = 2.0 ** -8 * np.abs(ref) + 2e-7 * np.abs(x)
    outs = {}
    for name, mode in MODES:
        _say(f"[gemm-gelu-range] mode={name}")
        _, _, _, out, _ = run_gemm(gi, m, n, k, mode)
        err = np.abs(out.astype(np.float64) - ref[None, :])
        assert (err <= bound[None, :]).all(), (err / np.maximum(bound, 1e-300)).max()
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


def test_gemm_full_size_sampled():
    """The benchmark shape 4096^3, checked on sampled elements one by one."""
    m = n = k = 4096
    _say("[gemm-full] generating")
    gi = gemm_inputs(seed=0, m=m, n=n, k=k)
    rng = np.random.default_rng(7)
    rows, cols = rng.integers(0, m, 3000), rng.integers(0, n, 3000)
    # every tile corner too
    rows = np.concatenate([rows, np.repeat(np.arange(0, m, 256), 16), np.repeat(np.arange(255, m, 256), 16)])
    cols = np.concatenate([cols, np.tile(np.arange(0, n, 256), 16), np.tile(np.arange(255, n, 256), 16)])
    ref = mathref.gemm_bias_gelu_at(gi.a, gi.bt, gi.bias, rows, cols)
    outs = {}
    for name, mode in MODES:
        _say(f"[gemm-full] mode={name}")
        _, _, _, out, _ = run_gemm(gi, m, n, k, mode)
        check_close(out[rows, cols], ref)
        outs[name] = out
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


def test_gemm_rejects_unsupported_shapes():
    prog = gemm_program(300, 256, 64)
    plan = Plan(prog)
    t = torch.zeros(16, dtype=torch.int32, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([t, t, t, t], t, t, 1)
    assert e.value.status == bfs.E_UNSUPPORTED


def test_gemm_watchdog():
    m, n, k = 256, 256, 64
    gi = gemm_inputs(seed=3, m=m, n=n, k=k)
    prog = gemm_program(m, n, k)
    plan = Plan(prog)
    tt = gemm_trips(m, n, k)
    trips, toff = trip_tensors(tt)
    a, bt = _bits_to_dev(gi.a), _bits_to_dev(gi.bt)
    bias = torch.from_numpy(gi.bias).cuda()
    c = torch.zeros(m * n, dtype=torch.int16, device="cuda")
    _say("[gemm-watchdog]")
    plan.run([a, bt, bias, c], trips, toff, tt.n_wg, watchdog_polls=2000, fault_dep=0, fault_delta=1 << 20)
    with pytest.raises(BfsError) as e:
        plan.status()
    assert e.value.status == bfs.E_DEADLOCK
    plan.run([a, bt, bias, c], trips, toff, tt.n_wg)
    plan.status()
