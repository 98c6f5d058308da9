"""The no-allocation entry point (bfs_run_noalloc) against bfs_run.

Each case calls bfs_run_noalloc through the C ABI twice in a row, the second
time on a smaller input, and requires outputs bit-identical to bfs_run's on
the same inputs (the two entry points launch the same kernels; only where
the plan's tables and error words live differs).  Interpreter plans read
their tables from the fixed device array, so interleaving two plans checks
that each launch sees its own tables."""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, BfsError, Plan, bfs  # noqa: E402
from tests.gpu_util import dev, trip_tensors  # noqa: E402
from workloads import (OP_NOP, ProgramBuilder, chain_workload, gemm_program, gemm_trips,  # noqa: E402
                       ring_workload, stream_workload)
from workloads.tensors import gemm_inputs  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bfs.lib()


def _say(*a):
    print(*a, flush=True, file=sys.stderr)


def _tile_run(w, plan, n_out, noalloc):
    trips, toff = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    out = torch.full((n_out,), float("nan"), dtype=torch.float32, device="cuda")
    run = plan.run_noalloc if noalloc else plan.run
    run([base, x, out], trips, toff, w.trips.n_wg)
    plan.status()
    return out.cpu().numpy()


@pytest.mark.parametrize("mode", [MODE_BARRIER_FREE, MODE_BARRIER])
def test_noalloc_interpreter_two_calls_and_interleaved_plans(mode):
    """Chain (16 outer iterations), then a smaller chain (5), then the ring
    program, then the first chain again: each equals bfs_run bit for bit."""
    cases = [("chain16", chain_workload(seed=0, kernel="interp"), 256),
             ("chain5", chain_workload(seed=1, outer=5, kernel="interp"), 256),
             ("ring", ring_workload(seed=2, outer=6, n_wg=3), 3 * 256)]
    plans = {name: Plan(w.prog, mode) for name, w, _ in cases}
    for name, w, n_out in cases + [cases[0]]:
        _say(f"[noalloc-interp] mode={mode} {name}")
        got = _tile_run(w, plans[name], n_out, noalloc=True)
        want = _tile_run(w, Plan(w.prog, mode), n_out, noalloc=False)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), name


def test_noalloc_stream_two_calls():
    """The stream family (error words only) at 256 workgroups, then at 16."""
    for n_wg, outer in ((256, 64), (16, 9)):
        w = stream_workload(seed=3, n_wg=n_wg, outer=outer)
        _say(f"[noalloc-stream] n_wg={n_wg}")
        got = _tile_run(w, Plan(w.prog), w.n_tiles * 64, noalloc=True)
        want = _tile_run(w, Plan(w.prog), w.n_tiles * 64, noalloc=False)
        assert np.array_equal(got.view(np.uint32), want.view(np.uint32))
        assert np.array_equal(got, w.x.reshape(-1) + np.float32(1.0))


def test_noalloc_gemm_two_calls():
    for m, n, k in ((512, 768, 256), (256, 256, 96)):
        gi = gemm_inputs(seed=4, m=m, n=n, k=k)
        tt = gemm_trips(m, n, k)
        trips, toff = trip_tensors(tt)
        a = torch.from_numpy(gi.a.view(np.int16)).cuda()
        bt = torch.from_numpy(gi.bt.view(np.int16)).cuda()
        bias = torch.from_numpy(gi.bias).cuda()
        outs = []
        for noalloc in (True, False):
            _say(f"[noalloc-gemm] {m}x{n}x{k} noalloc={noalloc}")
            plan = Plan(gemm_program(m, n, k))
            c = torch.full((m * n,), -1, dtype=torch.int16, device="cuda")
            (plan.run_noalloc if noalloc else plan.run)([a, bt, bias, c], trips, toff, tt.n_wg)
            plan.status()
            outs.append(c.cpu().numpy())
        assert np.array_equal(outs[0], outs[1])


def test_noalloc_reports_device_errors_then_recovers():
    """A wait that can never be met (raised threshold, short watchdog) is
    recorded in the fixed array's error words and reported by
    bfs_run_status; the next call runs cleanly."""
    w = chain_workload(seed=0, kernel="interp")
    plan = Plan(w.prog)
    trips, toff = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    out = torch.zeros(256, dtype=torch.float32, device="cuda")
    _say("[noalloc-watchdog]")
    plan.run_noalloc([base, x, out], trips, toff, 1, watchdog_polls=2000, fault_dep=0, fault_delta=1 << 20)
    with pytest.raises(BfsError) as e:
        plan.status()
    assert e.value.status == bfs.E_DEADLOCK
    got = _tile_run(w, plan, 256, noalloc=True)
    want = _tile_run(w, Plan(w.prog), 256, noalloc=False)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_noalloc_rejects_plan_beyond_the_array():
    """An interpreter plan whose tables exceed the fixed array is refused
    with BFS_E_RESOURCE before anything is launched."""
    b = ProgramBuilder("interp", n_engines=1)
    with b.loop("A"):
        for i in range(20000):
            b.instr(0, OP_NOP, name=f"N{i}")
    p = b.build()
    p.tile_elems = 64
    plan = Plan(p)
    t = torch.zeros(8, dtype=torch.int64, device="cuda")
    _say("[noalloc-too-big]")
    with pytest.raises(BfsError) as e:
        plan.run_noalloc([t, t, t], t.int(), t, 1)
    assert e.value.status == bfs.E_RESOURCE
