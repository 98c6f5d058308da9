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


def log_records(plan, log_words, n_wg, cap, per_wave=False):
    """{(wg, dep): sorted list of (instance, threshold, observed)}; with
    per_wave the key is (wg, wave, dep) (every wave of a multi-wave engine
    evaluates the same waits)."""
    per = parse_debug_log(log_words, n_wg, plan.n_waves, cap)
    out = {}
    for (wg, wave), ent in per.items():
        for dep, inst, thr, obs in ent.tolist():
            key = (wg, wave, dep) if per_wave else (wg, dep)
            out.setdefault(key, []).append((inst, thr, obs))
    for k in out:
        out[k].sort()
    return out


def compare_log_with_oracle(prog, plan, logs, recs_by_wg, mode, no_wait=()):
    """Every emitted wait's logged threshold equals the oracle's, bit-exact,
    and the observed counter was never below it.  mode "per_instr": a
    barrier-free plan with one counter per instruction, whose thresholds are
    the Eq. 1 counts.  Dependencies in ``no_wait`` (ordered by barriers)
    must log nothing.  mode "per_engine": one counter per producer engine,
    thresholds the per-engine counter values of the oracle."""
    key = {"barrier_free": "sem_thr", "barrier": "barrier_thr", "per_instr": "count_thr",
           "per_engine": "eng_thr"}[mode]
    n = 0
    for wg, recs in recs_by_wg.items():
        for d in range(len(prog.deps)):
            if d in no_wait:
                assert (wg, d) not in logs, (wg, d)
                continue
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


def compare_wave_logs_with_oracle(prog, plan, logs, recs_by_wg, mode):
    """Multi-wave engines: every wave of the consumer's engine logs the same
    waits, each equal to the oracle's threshold, observed never below it."""
    key = {"barrier_free": "sem_thr", "barrier": "barrier_thr", "per_instr": "count_thr"}[mode]
    engine_waves = {}
    w = 0
    for e, n in enumerate(plan.waves_per_engine):
        engine_waves[e] = list(range(w, w + n))
        w += n
    n = 0
    for wg, recs in recs_by_wg.items():
        for d, (p, c, k) in enumerate(prog.deps):
            r = recs[recs["dep"] == d]
            want = [(int(i), int(t)) for i, t in zip(r["instance"], r[key])]
            for wave in engine_waves[prog.instrs[c].engine]:
                got = logs.get((wg, wave, d), [])
                if mode == "barrier" and not got and all(t == 0 for _, t in want):
                    continue
                assert [(i, t) for i, t, _ in got] == want, (wg, wave, d)
                for i, t, obs in got:
                    assert t == 0 or obs >= t, (wg, wave, d, i, t, obs)
                n += len(got)
    return n


def compare_batched_log_with_oracle(prog, logs, recs_by_wg):
    """Logs of the batched loop (one entry per batch wait): every logged
    threshold equals the oracle's at the logged instance, bit-exact, the
    observed counter was never below it, and every consumer instance of the
    oracle's trace needs no more than the entry that covers it (the first
    logged instance at or after it: batches wait before their first
    instance issues, for the largest threshold among their instances)."""
    n = 0
    for wg, recs in recs_by_wg.items():
        for d in range(len(prog.deps)):
            r = recs[recs["dep"] == d]
            want = {int(i): int(t) for i, t in zip(r["instance"], r["sem_thr"])}
            got = logs.get((wg, d), [])
            assert got, (wg, d)
            inst = np.array([i for i, _, _ in got], np.int64)
            thr = np.array([t for _, t, _ in got], np.int64)
            assert (np.diff(inst) > 0).all(), (wg, d)
            for i, t, obs in got:
                assert i in want and want[i] == t, (wg, d, i, t, want.get(i))
                assert t == 0 or obs >= t, (wg, d, i, t, obs)
            oi = np.array(sorted(want), np.int64)
            ot = np.array([want[i] for i in oi], np.int64)
            cover = np.searchsorted(inst, oi, side="left")
            assert (cover < len(inst)).all(), (wg, d)
            assert (ot <= thr[cover]).all(), (wg, d)
            n += len(got)
    return n
