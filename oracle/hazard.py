"""Happens-before coverage of a dependency graph (CPU race check).

TEST INFRASTRUCTURE ONLY.

Given the oracle's sequential trace of one workgroup, every instruction
instance gets its read and write set (ring slots, accumulators, output tiles)
from the tile-machine semantics.  Happens-before is built from

  * each engine's own program order (an engine issues and retires in order,
    Section 3.2 and the retire rule of Appendix A.2), and
  * each satisfied wait: a consumer instance that waited for a counter to
    reach a value happens after the producer-engine instruction whose
    retirement brought the counter to that value, hence (in-order
    retirement) after everything earlier on that engine, and
  * in the barrier-based scheme, every barrier: everything before it happens
    before everything after it (Section 3.4); in the barrier-free scheme with
    the fallback of Section 5.2, the barrier at the end of every iteration of
    each loop in ``barrier_loops``.

A conflicting pair of accesses (same location, at least one write) on two
different engines must be ordered.  The trace order is a topological order of
happens-before when every requirement is already met at the consumer's
program-order position (the ``order_ok`` flag), which lets vector clocks be
filled in one pass.
"""
from __future__ import annotations

import struct
from collections import defaultdict

import numpy as np

from workloads import (OP_ADDC, OP_LOAD, OP_NOP, OP_SCALE_ACC, OP_STORE_ACC,
                       OP_STORE_RING)


def _slot(args, r, rhat):
    gen_loop, n_gen, pos_loop, per_gen = args[2], args[3], args[4], args[5]
    hi = ((int(r[gen_loop]) - 1) % n_gen) * per_gen if gen_loop >= 0 else 0
    lo = ((int(rhat[pos_loop]) - 1) % per_gen) if pos_loop >= 0 else 0
    return hi + lo


def accesses(prog, instr, r, rhat, wg=0, base=0):
    """(reads, writes) of one tile-machine instruction instance."""
    ins = prog.instrs[instr]
    a = ins.args
    op = ins.opcode
    reads, writes = [], []
    if op == OP_NOP:
        pass
    elif op == OP_LOAD:
        writes.append(("ring", a[1], _slot(a, r, rhat)))
        reads.append(("buf", a[0], base + int(r[a[6]]) - 1))
    elif op == OP_SCALE_ACC:
        reads.append(("ring", a[0], _slot(a, r, rhat)))
        reads.append(("acc", a[1]))
        writes.append(("acc", a[1]))
    elif op == OP_STORE_ACC:
        reads.append(("acc", a[0]))
        writes.append(("buf", a[1], wg))
    elif op == OP_ADDC:
        s = _slot(a, r, rhat)
        reads.append(("ring", a[0], s))
        writes.append(("ring", a[1], s))
    elif op == OP_STORE_RING:
        reads.append(("ring", a[0], _slot(a, r, rhat)))
        writes.append(("buf", a[1], base + int(r[a[6]]) - 1))
    return reads, writes


def _parents(prog):
    par = {}
    for l, items in enumerate(prog.body):
        for kind, bid in items:
            if kind == 0:
                for i in prog.blocks[bid]:
                    par[i] = l
    return par


def _ancestors(prog, l):
    out = {l}
    while prog.loop_parent[l] >= 0:
        l = prog.loop_parent[l]
        out.add(l)
    return out


def check(prog, res, mode="barrier_free", thresholds=None, barrier_loops=()):
    """Return a list of unordered conflicting pairs (empty = covered).

    ``res`` is an ``oracle.core.OracleResult``.  ``thresholds`` optionally
    overrides, per record of ``res.recs``, the value a consumer waited for
    (to test a planner's formulas or an injected mistake); by default the
    oracle's own requirement is used."""
    inst = res.inst
    n = len(inst)
    E = prog.n_engines
    par = _parents(prog)
    recs = res.recs
    thr = recs["sem_thr"] if mode == "barrier_free" else recs["barrier_thr"]
    if thresholds is not None:
        thr = np.asarray(thresholds)
    waits = defaultdict(list)   # (instr, instance) -> [(dep, value)]
    for i, rec in enumerate(recs):
        waits[(prog.deps[rec["dep"]][1], int(rec["instance"]))].append((int(rec["dep"]), int(thr[i])))

    seq = np.zeros(n, np.int64)
    vc = np.zeros((n, E), np.int64)          # vc[x][e]: engine-e prefix known to precede x
    last_on = [-1] * E
    n_on = [0] * E
    exec_idx = defaultdict(int)
    # producer lookup: (loop, engine, counter value) -> instance; and for the
    # barrier scheme (region, engine, ordinal) -> instance
    by_cnt = {}
    by_bord = {}
    region_join = np.zeros(E, np.int64)
    cur_region = inst["region"][0] if n else 0
    region_members = []
    # fallback barriers: an instance after the b-th barrier of loop S (b =
    # completed iterations of S) follows every instance before it
    fb = sorted(barrier_loops) if mode == "barrier_free" else []
    anc = {i: _ancestors(prog, par[i]) for i in par}
    fb_phase = {S: 0 for S in fb}
    fb_join = {S: np.zeros(E, np.int64) for S in fb}
    fb_members = {S: [] for S in fb}
    for x in range(n):
        ins_id = int(inst["instr"][x])
        e = int(inst["engine"][x])
        fb_vc = np.zeros(E, np.int64)
        for S in fb:
            b = int(res.r_snap[x][S]) - (1 if S in anc[ins_id] else 0)
            if b > fb_phase[S]:
                for y in fb_members[S]:
                    fb_join[S] = np.maximum(fb_join[S], vc[y])
                fb_members[S] = []
                fb_phase[S] = b
            fb_vc = np.maximum(fb_vc, fb_join[S])
            fb_members[S].append(x)
        if mode == "barrier" and inst["region"][x] != cur_region:
            # a barrier separates everything before from everything after
            for y in region_members:
                region_join = np.maximum(region_join, vc[y])
            region_members = []
            cur_region = inst["region"][x]
        base_vc = vc[last_on[e]].copy() if last_on[e] >= 0 else np.zeros(E, np.int64)
        if mode == "barrier":
            base_vc = np.maximum(base_vc, region_join)
        base_vc = np.maximum(base_vc, fb_vc)
        k = exec_idx[ins_id]
        exec_idx[ins_id] += 1
        for dep, val in waits.get((ins_id, k), []):
            if val <= 0:
                continue
            p = prog.deps[dep][0]
            pe = prog.instrs[p].engine
            if mode == "barrier_free":
                y = by_cnt.get((par[p], pe, val))
            else:
                y = by_bord.get((int(inst["region"][x]), pe, val))
            if y is None:
                # waiting for a value never reached earlier in program order
                return [("unreachable-wait", x, dep, val)]
            base_vc = np.maximum(base_vc, vc[y])
        n_on[e] += 1
        seq[x] = n_on[e]
        base_vc[e] = n_on[e]
        vc[x] = base_vc
        last_on[e] = x
        region_members.append(x)
        by_cnt[(par[ins_id], e, int(inst["cnt_after"][x]))] = x
        by_bord[(int(inst["region"][x]), e, int(inst["bord"][x]))] = x

    # conflicting cross-engine pairs must be ordered
    loc_acc = defaultdict(list)   # location -> [(x, is_write)]
    for x in range(n):
        rd, wr = accesses(prog, int(inst["instr"][x]), res.r_snap[x], res.rhat_snap[x])
        for l in rd:
            loc_acc[l].append((x, False))
        for l in wr:
            loc_acc[l].append((x, True))
    bad = []
    for loc, acc in loc_acc.items():
        for i in range(len(acc)):
            xa, wa = acc[i]
            for j in range(i + 1, len(acc)):
                xb, wb = acc[j]
                if not (wa or wb):
                    continue
                ea, eb = int(inst["engine"][xa]), int(inst["engine"][xb])
                if ea == eb:
                    continue
                a_, b_ = (xa, xb) if xa < xb else (xb, xa)
                if vc[b_][int(inst["engine"][a_])] < seq[a_]:
                    bad.append((loc, a_, b_))
    return bad


def f32(bits):
    return struct.unpack("<f", struct.pack("<i", bits))[0]
