"""ctypes binding of the C oracle (``bfs_oracle.c``).

TEST INFRASTRUCTURE ONLY: imported by the tests, the smoke check and the
benchmark's CPU-baseline leg; the GPU library never imports it.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "bfs_oracle.c")


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (plain C, no GPU)."""
    if force or not os.path.exists(_LIB_PATH):
        subprocess.check_call(["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-shared", "-fPIC",
                               "-o", _LIB_PATH, _SRC])
    return _LIB_PATH


class _Prog(C.Structure):
    _fields_ = [
        ("n_engines", C.c_int32), ("n_loops", C.c_int32), ("n_blocks", C.c_int32),
        ("n_instrs", C.c_int32), ("n_deps", C.c_int32),
        ("loop_parent", C.c_void_p), ("body_off", C.c_void_p), ("body_kind", C.c_void_p),
        ("body_id", C.c_void_p), ("block_off", C.c_void_p), ("block_instrs", C.c_void_p),
        ("instr_engine", C.c_void_p), ("instr_opcode", C.c_void_p), ("instr_args", C.c_void_p),
        ("deps", C.c_void_p), ("tile_elems", C.c_int32), ("n_rings", C.c_int32),
        ("n_accs", C.c_int32), ("ring_slots", C.c_void_p),
    ]


INST_DTYPE = np.dtype([("instr", np.int32), ("engine", np.int32), ("cnt_after", np.int64),
                       ("cnt_before", np.int64), ("region", np.int64), ("bord", np.int64),
                       ("ecnt_after", np.int64)])
REC_DTYPE = np.dtype([("dep", np.int32), ("instance", np.int32), ("count_thr", np.int64),
                      ("sem_thr", np.int64), ("barrier_thr", np.int64), ("r_P", np.int64),
                      ("r_S", np.int64), ("rhat_S", np.int64), ("order_ok", np.int32),
                      ("pad", np.int32), ("eng_thr", np.int64)])

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build(force=True)
        L = C.CDLL(_LIB_PATH)
        L.orc_count_instances.restype = C.c_int64
        L.orc_count_instances.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p]
        L.orc_run.restype = C.c_int
        L.orc_run.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p,
                              C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64,
                              C.c_void_p, C.c_int64, C.c_void_p, C.c_void_p]
        L.orc_values.restype = C.c_int
        L.orc_values.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p,
                                 C.c_void_p, C.c_void_p, C.c_int64]
        _lib = L
    return _lib


def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


class _ProgHandle:
    """Keeps the numpy arrays behind an orc_prog alive."""

    def __init__(self, prog):
        f = prog.flat()
        self.keep = {
            "loop_parent": _i32(f["loop_parent"]), "body_off": _i32(f["body_off"]),
            "body_kind": _i32(f["body_kind"] or [0]), "body_id": _i32(f["body_id"] or [0]),
            "block_off": _i32(f["block_off"]), "block_instrs": _i32(f["block_instrs"] or [0]),
            "instr_engine": _i32(f["instr_engine"] or [0]), "instr_opcode": _i32(f["instr_opcode"] or [0]),
            "instr_args": _i32(np.array(f["instr_args"] or [[0] * 8]).reshape(-1)),
            "deps": _i32(np.array(f["deps"] or [(0, 0, 0)]).reshape(-1)),
            "ring_slots": _i32(f["ring_slots"]),
        }
        k = self.keep
        n_rings = sum(1 for s in f["ring_slots"] if s > 0)
        self.s = _Prog(
            f["n_engines"], len(f["loop_parent"]), len(f["block_off"]) - 1, len(f["instr_engine"]),
            len(f["deps"]), k["loop_parent"].ctypes.data, k["body_off"].ctypes.data,
            k["body_kind"].ctypes.data, k["body_id"].ctypes.data, k["block_off"].ctypes.data,
            k["block_instrs"].ctypes.data, k["instr_engine"].ctypes.data, k["instr_opcode"].ctypes.data,
            k["instr_args"].ctypes.data, k["deps"].ctypes.data, f["tile_elems"], n_rings, f["n_accs"],
            k["ring_slots"].ctypes.data)
        self.n_loops = len(f["loop_parent"])
        self.n_engines = f["n_engines"]

    @property
    def ptr(self):
        return C.addressof(self.s)


@dataclass
class OracleResult:
    inst: np.ndarray        # INST_DTYPE [n_inst]
    r_snap: np.ndarray      # int32 [n_inst, n_loops]
    rhat_snap: np.ndarray   # int32 [n_inst, n_loops]
    recs: np.ndarray        # REC_DTYPE [n_recs]
    final_cnt: np.ndarray   # int64 [n_loops, n_engines]
    out: np.ndarray | None  # fp64 values (if data given)


def run(prog, trips, trip_off_wg, wg=0, base=None, x=None, out_len=0) -> OracleResult:
    """Sequential walk + brute-force thresholds for one workgroup."""
    L = lib()
    h = _ProgHandle(prog)
    trips = _i32(trips)
    toff = np.ascontiguousarray(np.asarray(trip_off_wg, dtype=np.int64))
    n = L.orc_count_instances(h.ptr, trips.ctypes.data, toff.ctypes.data)
    if n < 0:
        raise ValueError("oracle: program too large")
    inst = np.zeros(max(n, 1), INST_DTYPE)
    rs = np.zeros((max(n, 1), h.n_loops), np.int32)
    rh = np.zeros((max(n, 1), h.n_loops), np.int32)
    # one record per (dependency, consumer instance)
    cns_ids = [d[1] for d in prog.deps]
    rec_cap = 1
    if n > 0:
        L.orc_run(h.ptr, trips.ctypes.data, toff.ctypes.data, wg, None, None, None, 0,
                  inst.ctypes.data, rs.ctypes.data, rh.ctypes.data, n, None, 0,
                  C.byref(C.c_int64(0)), None)
        counts = np.bincount(inst["instr"][:n], minlength=len(prog.instrs))
        rec_cap = max(1, int(sum(counts[c] for c in cns_ids)))
    recs = np.zeros(rec_cap, REC_DTYPE)
    fin = np.zeros((h.n_loops, h.n_engines), np.int64)
    nrec = C.c_int64(0)
    out = None
    bptr = xptr = optr = None
    if x is not None:
        base = np.ascontiguousarray(base, dtype=np.int64)
        x = np.ascontiguousarray(x, dtype=np.float32)
        out = np.zeros(out_len, np.float64)
        bptr, xptr, optr = base.ctypes.data, x.ctypes.data, out.ctypes.data
    rc = L.orc_run(h.ptr, trips.ctypes.data, toff.ctypes.data, wg, bptr, xptr, optr, out_len,
                   inst.ctypes.data, rs.ctypes.data, rh.ctypes.data, max(n, 1), recs.ctypes.data,
                   rec_cap, C.byref(nrec), fin.ctypes.data)
    if rc != 0:
        raise RuntimeError(f"oracle failed: {rc}")
    return OracleResult(inst[:n], rs[:n], rh[:n], recs[:nrec.value], fin, out)


def values(prog, trips, trip_off, base, x, out_len) -> np.ndarray:
    """fp64 reference output of a tile-machine workload over all workgroups."""
    L = lib()
    h = _ProgHandle(prog)
    trips = _i32(trips)
    toff = np.ascontiguousarray(np.asarray(trip_off, dtype=np.int64))
    base = np.ascontiguousarray(base, dtype=np.int64)
    x = np.ascontiguousarray(x, dtype=np.float32)
    out = np.zeros(out_len, np.float64)
    rc = L.orc_values(h.ptr, trips.ctypes.data, toff.ctypes.data, toff.shape[0], base.ctypes.data,
                      x.ctypes.data, out.ctypes.data, out_len)
    if rc != 0:
        raise RuntimeError(f"oracle values failed: {rc}")
    return out


def linearized_records(prog, res, d):
    """EXTENSION, not in the paper: the requirements of dependency d when its
    offset counts iterations of the shared loop S across all of S's trips in
    the workgroup.  Brute force over the trace: a consumer instance whose
    monotone count of S is r needs every producer instance whose count of S
    is at most r - k (none if r - k <= 0); its semaphore threshold is the
    producer's per-loop counter right after the latest such instance (0 if
    none).  Returns the records of d (consumer-instance order) with
    count_thr and sem_thr replaced."""
    from oracle import cases
    p, c, k = prog.deps[d]
    S = cases.classify(prog, d)[1]
    inst = res.inst
    rS = res.r_snap[:, S].astype(np.int64)
    prod = np.nonzero(inst["instr"] == p)[0]
    cons = np.nonzero(inst["instr"] == c)[0]
    recs = res.recs[res.recs["dep"] == d].copy()
    assert len(recs) == len(cons)
    for j, x in enumerate(cons):
        target = rS[x] - k
        counted = [y for y in prod if rS[y] <= target] if target > 0 else []
        recs[j]["count_thr"] = len(counted)
        recs[j]["sem_thr"] = inst["cnt_after"][max(counted)] if counted else 0
        recs[j]["eng_thr"] = inst["ecnt_after"][max(counted)] if counted else 0
    return recs
