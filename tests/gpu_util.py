"""Helpers shared by the GPU tests: device copies of workload inputs and
debug-log comparison against the oracle's records."""
import numpy as np
import torch

from paper_2608_13757_amd import parse_debug_log


def dev(a, dtype=None):
    t = torch.from_numpy(np.ascontiguousarray(a))
    if dtype is not None:
        t = t.to(dtype)
    return t.cuda()


def trip_tensors(tt):
    trips, off = tt.flat()
    return dev(trips), dev(off)


def wave_engine_map(plan):
    """wave index -> engine for a plan's launch layout."""
    out = []
    for e, w in enumerate(plan.waves_per_engine):
        out.extend([e] * w)
    return out


def log_records(plan, log_words, n_wg, cap):
    """{(wg, dep): sorted list of (instance, threshold, observed)} over waves."""
    per = parse_debug_log(log_words, n_wg, plan.n_waves, cap)
    out = {}
    for (wg, _wave), ent in per.items():
        for dep, inst, thr, obs in ent.tolist():
            out.setdefault((wg, dep), []).append((inst, thr, obs))
    for k in out:
        out[k].sort()
    return out


def compare_log_with_oracle(prog, plan, logs, recs_by_wg, mode):
    """Every emitted wait's logged threshold equals the oracle's, bit-exact,
    and the observed counter was never below it."""
    key = "sem_thr" if mode == "barrier_free" else "barrier_thr"
    n = 0
    for wg, recs in recs_by_wg.items():
        for d in range(len(prog.deps)):
            r = recs[recs["dep"] == d]
            want = [(int(i), int(t)) for i, t in zip(r["instance"], r[key])]
            got = logs.get((wg, d), [])
            if mode == "barrier":
                # barrier mode emits only same-region waits
                if not got and all(t == 0 for _, t in want):
                    continue
            assert [(i, t) for i, t, _ in got] == want, (wg, d)
            for i, t, obs in got:
                assert t == 0 or obs >= t, (wg, d, i, t, obs)
            n += len(got)
    return n
