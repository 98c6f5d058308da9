"""GPU parity of the barrier fallback (Section 5.2 falling back to the
barrier scheme of Section 3.4) on the interpreter: a two-stage pipeline whose
ring dependencies are outside the allocatable cases, and random nests with
such dependencies.  Values equal the oracle's (the tile-machine sums in fp32
against fp64: |diff| <= 1e-5 on tiles of U(-1, 1) with at most 24 terms of
0.5 each), every semaphore wait logs the oracle's threshold bit-exactly, the
fallback dependencies log none, and the two modes give bit-identical
outputs."""
import copy
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from oracle import cases, core  # noqa: E402
from paper_2608_13757_amd import MODE_BARRIER, MODE_BARRIER_FREE, BfsError, Plan, bfs  # noqa: E402
from tests.gpu_util import compare_log_with_oracle, dev, log_records, trip_tensors  # noqa: E402
from workloads import lag_pipeline_workload, random_nest, stream_workload  # noqa: E402

pytestmark = pytest.mark.gpu

MODES = [("barrier_free", MODE_BARRIER_FREE), ("barrier", MODE_BARRIER)]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bfs.lib()


def _say(*a):
    print(*a, flush=True, file=sys.stderr)


def _fallback_deps(prog):
    return {d for d in range(len(prog.deps)) if cases.classify(prog, d)[0] == cases.FALLBACK}


@pytest.mark.parametrize("lag,ring", [(2, 3), (3, 5), (1, 2), (2, 6)])
def test_lag_pipeline_parity(lag, ring):
    n_wg = 96
    w = lag_pipeline_workload(seed=lag * 10 + ring, n_wg=n_wg, lag=lag, ring_slots=ring)
    trips, off = w.trips.flat()
    res = {wg: core.run(w.prog, trips, off[wg], wg, w.base, w.x, n_wg * 256) for wg in range(n_wg)}
    ref = core.values(w.prog, trips, off, w.base, w.x, n_wg * 256)
    t_trips, t_off = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    fb = _fallback_deps(w.prog)
    assert fb
    outs = {}
    cap = 64
    for name, mode in MODES:
        _say(f"[fallback-lag] lag={lag} ring={ring} mode={name}")
        plan = Plan(w.prog, mode, fallback=True)
        out = torch.zeros(n_wg * 256, dtype=torch.float32, device="cuda")
        log = torch.zeros(plan.debug_log_words(n_wg, cap), dtype=torch.int32, device="cuda")
        plan.run([base, x, out], t_trips, t_off, n_wg, debug_log=log, debug_capacity=cap)
        plan.status()
        got = out.cpu().numpy()
        assert np.abs(got - ref).max() <= 1e-5
        logs = log_records(plan, log.cpu().numpy().view(np.uint32), n_wg, cap)
        recs = {wg: res[wg].recs for wg in range(n_wg)}
        n = compare_log_with_oracle(w.prog, plan, logs, recs, name, no_wait=fb if name == "barrier_free" else ())
        if name == "barrier_free":
            # one STORE wait per workgroup, plus the CONS waits when LOAD->CONS is C3 (lag 1)
            n_cons = sum(len(res[wg].recs[res[wg].recs["dep"] == 0]) for wg in range(n_wg))
            assert n == n_wg + (n_cons if lag == 1 else 0)
        # uninstrumented launch: same output
        out2 = torch.zeros_like(out)
        plan.run([base, x, out2], t_trips, t_off, n_wg)
        plan.status()
        assert torch.equal(out, out2)
        outs[name] = got
    assert np.array_equal(outs["barrier_free"].view(np.uint32), outs["barrier"].view(np.uint32))


def test_random_nests_with_fallback():
    """Random nests keeping every satisfiable dependency: the allocatable
    waits log the oracle's thresholds, the fallback ones log nothing, and
    every launch completes."""
    checked = programs = 0
    for seed in range(150):
        prog, tt = random_nest(seed, max_trip=4 if seed % 2 else 3)
        prog = copy.deepcopy(prog)
        prog.deps = [d for j, d in enumerate(prog.deps) if cases.classify(prog, j)[0] != cases.ORDER]
        fb = _fallback_deps(prog)
        if not fb:
            continue
        trips, off = tt.flat()
        res = core.run(prog, trips, off[0], 0)
        plan = Plan(prog, fallback=True)
        t_trips, t_off = trip_tensors(tt)
        base = torch.zeros(1, dtype=torch.int64, device="cuda")
        x = torch.zeros(64, dtype=torch.float32, device="cuda")
        out = torch.zeros(64, dtype=torch.float32, device="cuda")
        cap = 256
        log = torch.zeros(plan.debug_log_words(1, cap), dtype=torch.int32, device="cuda")
        plan.run([base, x, out], t_trips, t_off, 1, debug_log=log, debug_capacity=cap)
        plan.status()
        logs = log_records(plan, log.cpu().numpy().view(np.uint32), 1, cap)
        checked += compare_log_with_oracle(prog, plan, logs, {0: res.recs}, "barrier_free", no_wait=fb)
        programs += 1
    assert programs > 40 and checked > 200


def test_fallback_plan_of_fused_family_unsupported():
    """A barrier-free plan of the stream family with a fallback dependency
    is refused at launch (only the interpreter executes the barriers)."""
    w = stream_workload(seed=0, n_wg=2, outer=3)
    prog = copy.deepcopy(w.prog)
    names = [i.name for i in prog.instrs]
    prog.deps = list(prog.deps) + [(names.index("LOAD"), names.index("MARK_O"), 2)]
    plan = Plan(prog, fallback=True)
    assert plan.stats()["n_fallback"] == 1
    t_trips, t_off = trip_tensors(w.trips)
    base, x = dev(w.base), dev(w.x)
    out = torch.zeros(w.x.size, dtype=torch.float32, device="cuda")
    with pytest.raises(BfsError) as e:
        plan.run([base, x, out], t_trips, t_off, w.trips.n_wg)
    assert e.value.status == bfs.E_UNSUPPORTED
