"""GPU parity of the AdamW family (load / vector / store engines over a loop
of parameter chunks, updated in place in an LDS ring slot).

The kernel computes in fp32 from fp32 state and the program's fp32
hyperparameters, the oracle in fp64 from the same values.  Bound per
element, from the operations' rounding (u = 2^-24, four roundings each):
|dm| <= 4u (b1|m| + (1-b1)|g|), |dv| <= 4u (b2 v + (1-b2) g^2), and for p'
the propagation of those through r = c1 m' / (sqrt(c2 v') + eps):
|dp| <= 4u (|p| + lr |update|) + lr (c1 |dm| / den + |r| (4u + c2 |dv| /
(2 sqrt(c2 v') den))); every output is also within the 1e-5 max-abs bar of
fp32 stages.  Thresholds bit-exact against the oracle's brute force; both
modes give bit-identical outputs."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import core  # noqa: E402
from oracle.mathref import adamw_step  # noqa: E402
from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, BfsError, Plan, bfs  # noqa: E402
from tests.gpu_util import compare_wave_logs_with_oracle, log_records  # noqa: E402
from workloads import ADAM_HP, adamw_default_wg, adamw_program, adamw_worklist  # noqa: E402
from workloads.tensors import AdamInputs, adamw_inputs  # noqa: E402

pytestmark = pytest.mark.gpu

MODES = [("barrier_free", MODE_BARRIER_FREE), ("barrier", MODE_BARRIER)]
U = 2.0 ** -24


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bfs.lib()


def _say(*a):
    print(*a, flush=True, file=sys.stderr)


def run_adam(ai, n_wg, mode, chunk=1024, waves=2, ring=2, cap=0, **kw):
    n = ai.p.size
    hp = ADAM_HP
    prog = adamw_program(n, chunk, waves, ring, hp["lr"], hp["b1"], hp["b2"], hp["eps"], hp["wd"], hp["t"])
    plan = Plan(prog, mode)
    base, tt = adamw_worklist(n, chunk, n_wg)
    t_np, o_np = tt.flat()
    P, G, M, V = (torch.from_numpy(a.copy()).cuda() for a in (ai.p, ai.g, ai.m, ai.v))
    log = None
    if cap:
        log = torch.zeros(plan.debug_log_words(n_wg, cap), dtype=torch.int32, device="cuda")
    plan.run([torch.from_numpy(base).cuda(), P, G, M, V], torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda(),
             n_wg, debug_log=log, debug_capacity=cap, **kw)
    plan.status()
    logs = log.cpu().numpy().view(np.uint32) if cap else None
    return prog, plan, tt, P.cpu().numpy(), M.cpu().numpy(), V.cpu().numpy(), logs


def check(ai, p, m, v):
    # the program carries the hyperparameters as fp32 values: those are the
    # ones the step is defined with
    hp = {k: (float(np.float32(x)) if k != "t" else x) for k, x in ADAM_HP.items()}
    b1, b2, lr, eps, wd, t = hp["b1"], hp["b2"], hp["lr"], hp["eps"], hp["wd"], hp["t"]
    p0, g, m0, v0 = (a.astype(np.float64) for a in (ai.p, ai.g, ai.m, ai.v))
    rp, rm, rv = adamw_step(p0, g, m0, v0, lr, b1, b2, eps, wd, t)
    c1, c2 = 1.0 / (1.0 - b1 ** t), 1.0 / (1.0 - b2 ** t)
    tol_m = 4 * U * (b1 * np.abs(m0) + (1 - b1) * np.abs(g))
    tol_v = 4 * U * (b2 * v0 + (1 - b2) * g * g)
    den = np.sqrt(c2 * rv) + eps
    r = c1 * rm / den
    upd = r + wd * p0
    tol_r = c1 * tol_m / den + np.abs(r) * (4 * U + c2 * tol_v / (2 * np.sqrt(c2 * rv) * den + 1e-300))
    tol_p = 4 * U * (np.abs(p0) + lr * np.abs(upd)) + lr * tol_r
    for got, ref, tol, name in ((m, rm, tol_m, "m"), (v, rv, tol_v, "v"), (p, rp, tol_p, "p")):
        d = np.abs(got.astype(np.float64) - ref)
        assert d.max() <= 1e-5, name
        bad = d > tol
        assert not bad.any(), (name, np.argwhere(bad)[:5].ravel(), d[bad][:5], tol[bad][:5])


@pytest.mark.parametrize("n,chunk,waves,ring,n_wg", [
    (4096, 1024, 2, 2, 3),        # ragged chunk runs over 3 workgroups
    (4004, 256, 1, 2, 5),         # a partial last chunk
    (12, 256, 1, 1, 2),           # fewer parameters than a chunk, an empty trip
    (65536, 512, 4, 3, 7),        # four vector waves, three slots
    (8192, 1024, 2, 4, 40),       # more workgroups than chunks
])
def test_adamw_small_parity_and_thresholds(n, chunk, waves, ring, n_wg):
    ai = adamw_inputs(seed=n + chunk, n=n)
    outs = {}
    for name, mode in MODES:
        _say(f"[adamw] n={n} chunk={chunk} waves={waves} ring={ring} n_wg={n_wg} mode={name}")
        prog, plan, tt, p, m, v, logw = run_adam(ai, n_wg, mode, chunk, waves, ring, cap=64)
        check(ai, p, m, v)
        trips, off = tt.flat()
        recs = {wg: core.run(prog, trips, off[wg], wg).recs for wg in range(n_wg)}
        logs = log_records(plan, logw, n_wg, 64, per_wave=True)
        cnt = compare_wave_logs_with_oracle(prog, plan, logs, recs, name)
        assert name == "barrier" or cnt > 0
        _, _, _, p2, m2, v2, _ = run_adam(ai, n_wg, mode, chunk, waves, ring)
        assert all(np.array_equal(a.view(np.uint32), b.view(np.uint32)) for a, b in ((p, p2), (m, m2), (v, v2)))
        outs[name] = (p, m, v)
    for a, b in zip(outs["barrier_free"], outs["barrier"]):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_adamw_zero_gradient_and_moments():
    n = 2048
    ai = adamw_inputs(seed=9, n=n)
    z = np.zeros(n, np.float32)
    zi = AdamInputs(ai.p, z, z, z)
    for name, mode in MODES:
        _say(f"[adamw-zero] mode={name}")
        _, _, _, p, m, v, _ = run_adam(zi, 2, mode)
        check(zi, p, m, v)
        assert not m.any() and not v.any()


@pytest.mark.parametrize("n_wg", [adamw_default_wg(1 << 20), 256], ids=["bench", "wg256"])
def test_adamw_full_size(n_wg):
    """2^20 parameters at the benchmark's launch shape (512 workgroups of 2
    chunks of 1024), then 256 workgroups of 4 chunks; every element against
    the oracle; the modes agree."""
    ai = adamw_inputs(seed=0)
    outs = {}
    for name, mode in MODES:
        _say(f"[adamw-full] n_wg={n_wg} mode={name}")
        _, _, _, p, m, v, _ = run_adam(ai, n_wg, mode)
        check(ai, p, m, v)
        outs[name] = (p, m, v)
    for a, b in zip(outs["barrier_free"], outs["barrier"]):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_adamw_watchdog():
    ai = adamw_inputs(seed=4, n=8192)
    _say("[adamw-watchdog]")
    with pytest.raises(BfsError) as e:
        run_adam(ai, 2, MODE_BARRIER_FREE, watchdog_polls=2000, fault_dep=0, fault_delta=1 << 20)
    assert e.value.status == bfs.E_DEADLOCK
    run_adam(ai, 2, MODE_BARRIER_FREE)


def test_adamw_chunks_beyond_input_rejected():
    n = 4096
    ai = adamw_inputs(seed=5, n=n)
    prog = adamw_program(n, 1024)
    plan = Plan(prog)
    base, tt = adamw_worklist(n, 1024, 2)
    tt.per_wg[1][1][0] += 2
    t_np, o_np = tt.flat()
    P, G, M, V = (torch.from_numpy(a.copy()).cuda() for a in (ai.p, ai.g, ai.m, ai.v))
    _say("[adamw-bad-trip]")
    plan.run([torch.from_numpy(base).cuda(), P, G, M, V], torch.from_numpy(t_np).cuda(), torch.from_numpy(o_np).cuda(), 2)
    with pytest.raises(BfsError) as e:
        plan.status()
    assert e.value.status == bfs.E_INVALID


def test_adamw_rejects_unsupported_shapes():
    for n, chunk, waves in ((1001, 1024, 2), (4096, 300, 2), (4096, 1024, 3)):
        plan = Plan(adamw_program(n, chunk, waves))
        t = torch.zeros(16, dtype=torch.int64, device="cuda")
        with pytest.raises(BfsError) as e:
            plan.run([t, t, t, t, t], t.int(), t, 1)
        assert e.value.status == bfs.E_UNSUPPORTED
