"""GPU parity of the RMSNorm + FP8 quantization family (load / vector /
store engines over a software-pipelined row loop).

Scales are fp32: |gpu - oracle| <= 1e-5 absolute and <= 2e-5 relative to the
fp64 oracle.  Codes are compared exactly, except where the oracle's y / s
lies within a relative 2^-18 of a rounding midpoint between two E4M3 values:
there either neighbour is a correct rounding (the kernel's fp32 evaluation
of y / s is within a few ulp, 2^-21 relative, of the exact value).
Thresholds are bit-exact against the oracle's brute force for every wave of
every consumer engine; both modes give bit-identical outputs."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import core, mathref  # noqa: E402
from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, BfsError, Plan, bfs  # noqa: E402
from tests.gpu_util import compare_wave_logs_with_oracle, log_records  # noqa: E402
from workloads import rmsnorm_program, rmsnorm_worklist  # noqa: E402
from workloads.tensors import rmsnorm_inputs, to_bf16_bits  # noqa: E402

pytestmark = pytest.mark.gpu

MODES = [("barrier_free", MODE_BARRIER_FREE), ("barrier", MODE_BARRIER)]
EPS = 1e-6


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bfs.lib()


def _say(*a):
    print(*a, flush=True, file=sys.stderr)


def run_rms(x_bits, g_bits, n_wg, mode, waves=4, nx=2, nq=2, cap=0, **kw):
    t, h = x_bits.shape
    prog = rmsnorm_program(t, h, waves, nx, nq, EPS)
    plan = Plan(prog, mode)
    base_np, tt = rmsnorm_worklist(t, n_wg)
    t_np, o_np = tt.flat()
    X = torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).cuda()
    G = torch.from_numpy(np.ascontiguousarray(g_bits).view(np.int16)).cuda()
    Q = torch.full((t * h,), 0x7F, dtype=torch.uint8, device="cuda")
    S = torch.full((t,), -1.0, dtype=torch.float32, device="cuda")
    log = None
    if cap:
        log = torch.zeros(plan.debug_log_words(n_wg, cap), dtype=torch.int32, device="cuda")
    plan.run([torch.from_numpy(base_np).cuda(), X, G, Q, S], torch.from_numpy(t_np).cuda(),
             torch.from_numpy(o_np).cuda(), n_wg, debug_log=log, debug_capacity=cap, **kw)
    plan.status()
    logs = log.cpu().numpy().view(np.uint32) if cap else None
    return prog, plan, tt, Q.cpu().numpy().reshape(t, h), S.cpu().numpy(), logs


def check_rows(codes, scales, x_bits, g_bits, rows):
    ref_c, ref_s, ref_t = mathref.rmsnorm_fp8_rows(x_bits, g_bits, EPS, rows)
    got_c, got_s = codes[rows], scales[rows].astype(np.float64)
    assert np.max(np.abs(got_s - ref_s)) <= 1e-5
    assert np.max(np.abs(got_s - ref_s) / ref_s) <= 2e-5
    amb = mathref.e4m3fn_ambiguous(ref_t)
    exact = ~amb
    assert np.array_equal(got_c[exact], ref_c[exact]), np.argwhere((got_c != ref_c) & exact)[:5]
    lo = mathref.e4m3fn_encode(ref_t[amb] * (1 - 2.0 ** -18))
    hi = mathref.e4m3fn_encode(ref_t[amb] * (1 + 2.0 ** -18))
    assert np.all((got_c[amb] == lo) | (got_c[amb] == hi))
    return int(amb.sum())


@pytest.mark.parametrize("t,h,n_wg,waves,nx,nq", [
    (96, 8192, 5, 4, 2, 2),       # ragged split over 5 workgroups
    (150, 1024, 7, 1, 1, 1),      # single-slot rings, one vector wave
    (128, 2048, 9, 2, 3, 2),      # two vector waves
    (64, 4096, 3, 8, 2, 1),       # eight vector waves
    (40, 8192, 6, 8, 4, 4),       # four-slot rings
    (20, 1024, 32, 2, 2, 2),      # more workgroups than rows: empty trips
])
def test_rms_small_parity_and_thresholds(t, h, n_wg, waves, nx, nq):
    ri = rmsnorm_inputs(seed=t + h, t=t, h=h)
    outs = {}
    for name, mode in MODES:
        _say(f"[rms] t={t} h={h} n_wg={n_wg} waves={waves} rings={nx},{nq} mode={name}")
        prog, plan, tt, q, s, logw = run_rms(ri.x, ri.gamma, n_wg, mode, waves, nx, nq, cap=256)
        check_rows(q, s, ri.x, ri.gamma, np.arange(t))
        trips, off = tt.flat()
        recs = {wg: core.run(prog, trips, off[wg], wg).recs for wg in range(n_wg)}
        logs = log_records(plan, logw, n_wg, 256, per_wave=True)
        n = compare_wave_logs_with_oracle(prog, plan, logs, recs, name)
        assert name == "barrier" or n > 0
        # uninstrumented launch: same outputs
        _, _, _, q2, s2, _ = run_rms(ri.x, ri.gamma, n_wg, mode, waves, nx, nq)
        assert np.array_equal(q, q2) and np.array_equal(s.view(np.uint32), s2.view(np.uint32))
        outs[name] = (q, s)
    assert np.array_equal(outs["barrier_free"][0], outs["barrier"][0])
    assert np.array_equal(outs["barrier_free"][1].view(np.uint32), outs["barrier"][1].view(np.uint32))


def test_rms_special_rows():
    """A zero row (scale 1, codes 0), a constant row, one huge outlier, and a
    row of tiny values (subnormal codes)."""
    t, h = 8, 1024
    rng = np.random.default_rng(5)
    x = rng.standard_normal((t, h)).astype(np.float32)
    x[0] = 0
    x[1] = -1.5
    x[2, 17] = 3e4
    x[3] = rng.standard_normal(h).astype(np.float32) * 1e-3
    x[3, 5] = 1.0
    xb = to_bf16_bits(x)
    gb = to_bf16_bits(np.ones(h, np.float32))
    for name, mode in MODES:
        _say(f"[rms-special] mode={name}")
        _, _, _, q, s, _ = run_rms(xb, gb, 3, mode, waves=2)
        check_rows(q, s, xb, gb, np.arange(t))
        assert s[0] == 1.0 and not q[0].any()
        assert np.all(q[1] == 0xFE)
        assert q[2, 17] == 0x7E and np.count_nonzero(q[3] & 0x78 == 0) > 0


def test_rms_full_size_sampled():
    """32768 x 8192 at the benchmark's launch shape (768 workgroups, four
    vector waves, double-buffered rings): 256 sampled rows against the oracle;
    every nonzero row reaches the largest code; the modes agree."""
    ri = rmsnorm_inputs(seed=0)
    rows = np.sort(np.random.default_rng(11).choice(ri.x.shape[0], 256, replace=False))
    outs = {}
    for name, mode in MODES:
        _say(f"[rms-full] mode={name}")
        _, _, _, q, s, _ = run_rms(ri.x, ri.gamma, 768, mode)
        amb = check_rows(q, s, ri.x, ri.gamma, rows)
        assert amb < 0.001 * rows.size * ri.x.shape[1]
        assert np.all(np.max(q & 0x7F, axis=1) == 0x7E)
        outs[name] = (q, s)
    assert np.array_equal(outs["barrier_free"][0], outs["barrier"][0])
    assert np.array_equal(outs["barrier_free"][1].view(np.uint32), outs["barrier"][1].view(np.uint32))


def test_rms_watchdog():
    ri = rmsnorm_inputs(seed=2, t=32, h=1024)
    _say("[rms-watchdog]")
    with pytest.raises(BfsError) as e:
        run_rms(ri.x, ri.gamma, 4, MODE_BARRIER_FREE, waves=2, watchdog_polls=2000, fault_dep=0,
                fault_delta=1 << 20)
    assert e.value.status == bfs.E_DEADLOCK
    run_rms(ri.x, ri.gamma, 4, MODE_BARRIER_FREE, waves=2)


def test_rms_rows_beyond_input_rejected():
    """A trip table that runs past the last row is reported, not executed."""
    t, h = 16, 1024
    ri = rmsnorm_inputs(seed=4, t=t, h=h)
    prog = rmsnorm_program(t, h, waves=2)
    plan = Plan(prog)
    base_np, tt = rmsnorm_worklist(t, 2)
    tt.per_wg[1][1][0] += 3
    t_np, o_np = tt.flat()
    X = torch.from_numpy(ri.x.view(np.int16)).cuda()
    G = torch.from_numpy(ri.gamma.view(np.int16)).cuda()
    Q = torch.zeros(t * h, dtype=torch.uint8, device="cuda")
    S = torch.zeros(t, dtype=torch.float32, device="cuda")
    _say("[rms-bad-trip]")
    plan.run([torch.from_numpy(base_np).cuda(), X, G, Q, S], torch.from_numpy(t_np).cuda(),
             torch.from_numpy(o_np).cuda(), 2)
    with pytest.raises(BfsError) as e:
        plan.status()
    assert e.value.status == bfs.E_INVALID


def test_rms_rejects_unsupported_shapes():
    for h, waves in ((1000, 1), (16384, 4), (8192, 1), (1024, 4)):
        prog = rmsnorm_program(64, h, waves)
        plan = Plan(prog)
        t = torch.zeros(16, dtype=torch.int64, device="cuda")
        with pytest.raises(BfsError) as e:
            plan.run([t, t, t, t, t], t.int(), t, 1)
        assert e.value.status == bfs.E_UNSUPPORTED
