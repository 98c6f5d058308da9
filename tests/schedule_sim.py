"""Schedule exploration of the specification and implementation transition
systems of the paper's appendix (specification steps Issue / Commit /
Retire, Appendix A.2; implementation with semaphore checks at issue and
increments at retirement, Appendix A.4), over one workgroup of a program.

TEST INFRASTRUCTURE ONLY: used by the tests; the GPU library never imports
it.

The specification issues an instruction instance when every dependency it
consumes is satisfied: the producer has retired at least the Eq. 1 count of
times (the oracle's brute force).  The implementation issues it when every
semaphore the plan assigns to those dependencies holds at least the plan's
threshold, evaluated through the library's ``bfs_eval_threshold`` on the
consumer engine's loop registers at that instance (the oracle's register
snapshot), and increments, at each retirement, the semaphores the
instruction updates.  Both systems take the same random steps: at every
reachable state the two issue predicates must agree for every engine's next
instruction (every wait fires if and only if its dependency is satisfied:
safety and liveness), every schedule must run to completion, and the final
datapath state must equal the sequential one.

Dependencies of a plan's barrier fallback (Section 5.2) have no semaphore:
the implementation orders them by a barrier at the end of every iteration of
their shared loop S, after which an engine issues nothing until every
instance of the earlier iterations of S, on every engine, has retired.  For
those only safety is required (a barrier may hold back an instance whose
dependency is met).

Datapath operations are opaque, as in the paper's model: an instance's
commit reads the cells of its read set (the tile-machine semantics of
``oracle.hazard.accesses``) and writes, to each cell of its write set, a
value determined by its identity and the values it read.  An engine's
in-flight instances may commit in any order except that one does not pass an
older instance of the same engine whose accesses conflict with its own (a
GPU wave's accesses to its own data take effect in program order).
"""
from __future__ import annotations

import random
from dataclasses import dataclass

from oracle import core, hazard


@dataclass
class Outcome:
    ok: bool
    kind: str = ""          # "", "unsafe", "blocked", "deadlock", "values"
    detail: str = ""
    steps: int = 0


def _parents(prog):
    par = {}
    for l, items in enumerate(prog.body):
        for kind, bid in items:
            if kind == 0:
                for i in prog.blocks[bid]:
                    par[i] = l
    return par


def _listing(prog):
    """Instructions of each loop body in listing order."""
    order = {}
    for l, items in enumerate(prog.body):
        seq = []
        for kind, bid in items:
            if kind == 0:
                seq += list(prog.blocks[bid])
        order[l] = seq
    return order


class Model:
    """One workgroup's instances, their requirements under both systems and
    their datapath accesses.  ``threshold_delta`` maps a dependency to an
    amount added to the implementation's threshold, ``drop_updates`` lists
    (instruction, counter) increments the implementation omits: planted
    mistakes for the tests of this simulator."""

    def __init__(self, prog, plan, trips, trip_off_wg, wg=0, per_instr=False, threshold_delta=None,
                 drop_updates=(), barrier_loops=None):
        res = core.run(prog, trips, trip_off_wg, wg)
        self.prog = prog
        inst = res.inst
        self.n = n = len(inst)
        self.instr = [int(x) for x in inst["instr"]]
        self.engine = [int(x) for x in inst["engine"]]
        self.n_engines = prog.n_engines
        self.seq = [[i for i in range(n) if self.engine[i] == e] for e in range(self.n_engines)]
        # occurrence number of every instance among its instruction's instances
        occ, seen = [0] * n, {}
        for i in range(n):
            occ[i] = seen.get(self.instr[i], 0)
            seen[self.instr[i]] = occ[i] + 1
        by_occ = {(self.instr[i], occ[i]): i for i in range(n)}
        all_formulas = {f["dep"]: f for f in plan.formulas()}
        formulas = {d: f for d, f in all_formulas.items() if f["kase"] != 4}
        if barrier_loops is None:
            barrier_loops = sorted({f["loop_S"] for f in all_formulas.values() if f["kase"] == 4} - {0})
        self.barrier_loops = list(barrier_loops)
        delta = threshold_delta or {}
        # requirements: instance -> [(dep, producer instr, Eq. 1 count, counter, implementation threshold)];
        # fallback dependencies: instance -> [(dep, producer instr, Eq. 1 count)]
        self.req = [[] for _ in range(n)]
        self.req_fb = [[] for _ in range(n)]
        for rec in res.recs:
            d = int(rec["dep"])
            prd, cns, _k = prog.deps[d]
            i = by_occ[(cns, int(rec["instance"]))]
            if d not in formulas:
                self.req_fb[i].append((d, prd, int(rec["count_thr"])))
                continue
            f = formulas[d]
            thr = plan.eval_threshold(d, int(rec["r_P"]), int(rec["rhat_S"])) + delta.get(d, 0)
            self.req[i].append((d, prd, int(rec["count_thr"]), f["counter"], max(thr, 0)))
        # semaphores each instruction increments at retirement
        par = _parents(prog)
        self.updates = {i: [] for i in range(len(prog.instrs))}
        self.counters = sorted({f["counter"] for f in formulas.values()})
        if per_instr:
            for d, f in formulas.items():
                prd = prog.deps[d][0]
                if f["counter"] not in self.updates[prd]:
                    self.updates[prd].append(f["counter"])
        else:
            key = {}
            for f in formulas.values():
                key[(f["loop_P"], f["prd_engine"])] = f["counter"]
            for i, ins in enumerate(prog.instrs):
                c = key.get((par[i], ins.engine))
                if c is not None:
                    self.updates[i].append(c)
        for i, c in drop_updates:
            self.updates[i] = [x for x in self.updates[i] if x != c]
        # barrier phase of every instance per barrier loop S: the iterations
        # of S completed before it (r_S, less the one it runs in)
        def inside(i, S):
            l = par[i]
            while l >= 0:
                if l == S:
                    return True
                l = prog.loop_parent[l]
            return False
        self.phase = [[int(res.r_snap[x][S]) - inside(self.instr[x], S) for S in self.barrier_loops]
                      for x in range(n)]
        # instances that precede barrier b of loop j: need[j][b]
        self.need = []
        for j in range(len(self.barrier_loops)):
            top = max((ph[j] for ph in self.phase), default=0)
            cnt = [0] * (top + 2)
            for ph in self.phase:
                cnt[ph[j] + 1] += 1
            for b in range(1, len(cnt)):
                cnt[b] += cnt[b - 1]
            self.need.append(cnt)        # cnt[b] = instances with phase < b
        # datapath accesses of every instance
        self.reads, self.writes = [], []
        for i in range(n):
            rd, wr = hazard.accesses(prog, self.instr[i], res.r_snap[i], res.rhat_snap[i], wg)
            self.reads.append(rd)
            self.writes.append(wr)

    def conflict(self, a, b):
        wa, wb = set(self.writes[a]), set(self.writes[b])
        return bool(wa & wb or wa & set(self.reads[b]) or wb & set(self.reads[a]))

    def commit(self, data, i):
        vals = tuple(data.get(c, 0) for c in self.reads[i])
        for c in self.writes[i]:
            data[c] = hash((i,) + vals)

    def sequential(self):
        data = {}
        for i in range(self.n):
            self.commit(data, i)
        return data


def explore(model: Model, seed: int, issue_bias: float = 0.5) -> Outcome:
    """One random schedule of both systems, checked at every state."""
    rng = random.Random(seed)
    pos = [0] * model.n_engines
    ifl = [[] for _ in range(model.n_engines)]       # [instance, committed]
    rc = {}                                          # retirements per instruction (specification)
    sema = {c: 0 for c in model.counters}            # semaphores (implementation)
    retired_ph = [{} for _ in model.barrier_loops]   # retired instances per barrier phase
    data = {}
    steps = 0

    def barriers_passed(i):
        for j, cnt in enumerate(model.need):
            b = model.phase[i][j]
            if sum(v for ph, v in retired_ph[j].items() if ph < b) < cnt[b]:
                return False
        return True

    while True:
        issue, other = [], []
        for e in range(model.n_engines):
            if pos[e] < len(model.seq[e]):
                i = model.seq[e][pos[e]]
                spec = all(rc.get(prd, 0) >= cnt for _, prd, cnt, _, _ in model.req[i])
                impl = all(sema[c] >= thr for _, _, _, c, thr in model.req[i])
                if impl and not spec:
                    return Outcome(False, "unsafe", f"engine {e} instance {i} issues before its dependency", steps)
                if spec and not impl:
                    return Outcome(False, "blocked", f"engine {e} instance {i} waits with its dependency met",
                                   steps)
                if impl and barriers_passed(i):
                    if not all(rc.get(prd, 0) >= cnt for _, prd, cnt in model.req_fb[i]):
                        return Outcome(False, "unsafe",
                                       f"engine {e} instance {i} passes its barriers before a fallback dependency",
                                       steps)
                    issue.append(e)
            for j, (i, done) in enumerate(ifl[e]):
                if not done and not any(not d2 and model.conflict(i2, i) for i2, d2 in ifl[e][:j]):
                    other.append(("commit", e, j))
            if ifl[e] and ifl[e][0][1]:
                other.append(("retire", e, 0))
        if not issue and not other:
            if any(pos[e] < len(model.seq[e]) for e in range(model.n_engines)):
                return Outcome(False, "deadlock", f"positions {pos}", steps)
            break
        steps += 1
        if issue and (not other or rng.random() < issue_bias):
            e = rng.choice(issue)
            ifl[e].append([model.seq[e][pos[e]], False])
            pos[e] += 1
            continue
        kind, e, j = rng.choice(other)
        if kind == "commit":
            model.commit(data, ifl[e][j][0])
            ifl[e][j][1] = True
        else:
            i = ifl[e].pop(0)[0]
            rc[model.instr[i]] = rc.get(model.instr[i], 0) + 1
            for j in range(len(model.barrier_loops)):
                b = model.phase[i][j]
                retired_ph[j][b] = retired_ph[j].get(b, 0) + 1
            for c in model.updates[model.instr[i]]:
                sema[c] += 1
    if data != model.sequential():
        return Outcome(False, "values", "final datapath state differs from the sequential one", steps)
    return Outcome(True, steps=steps)
