"""ctypes binding of libbfs (include/bfs.h): argument marshalling only.

Every computation on the hot path runs in the library's HIP kernels; this
module converts a program description into the C structs, holds plans, and
forwards device pointers (torch tensors or raw integers) and HIP streams.
Loading fails loudly when libbfs.so has not been built.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libbfs.so")

OK, E_INVALID, E_ORDER, E_NOT_ALLOCATABLE, E_RESOURCE, E_DEVICE, E_DEADLOCK, E_UNSUPPORTED = range(8)
MODE_BARRIER_FREE, MODE_BARRIER = 0, 1
ALLOC_PER_LOOP, ALLOC_PER_INSTR, ALLOC_PER_ENGINE = 0, 1, 2
PLAN_BARRIER_FALLBACK = 1
KASE_FALLBACK = 4
KERNELS = {"interp": 0, "stream3": 1, "gemm": 2, "attn": 3, "moe": 4, "rmsnorm": 5, "adamw": 6, "chain": 7}

EXPORTED = ["bfs_plan_create", "bfs_plan_formulas", "bfs_plan_static_waits", "bfs_plan_stats",
            "bfs_eval_threshold", "bfs_plan_destroy", "bfs_run", "bfs_run_noalloc", "bfs_run_status",
            "bfs_status_string", "bfs_last_error"]


class BfsError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{msg} (status {status})")
        self.status = status


class _Program(C.Structure):
    _fields_ = [
        ("kernel", C.c_int32), ("n_engines", C.c_int32), ("waves_per_engine", C.c_int32 * 8),
        ("n_loops", C.c_int32), ("loop_parent", C.c_void_p), ("loop_is_cond", C.c_void_p),
        ("body_off", C.c_void_p), ("body_kind", C.c_void_p), ("body_id", C.c_void_p),
        ("n_blocks", C.c_int32), ("block_off", C.c_void_p), ("block_instrs", C.c_void_p),
        ("n_instrs", C.c_int32), ("instr_engine", C.c_void_p), ("instr_opcode", C.c_void_p),
        ("instr_args", C.c_void_p), ("n_deps", C.c_int32), ("deps", C.c_void_p),
        ("tile_elems", C.c_int32), ("ring_slots", C.c_int32 * 4), ("n_accs", C.c_int32),
        ("dep_linear", C.c_void_p),
    ]


class Formula(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("dep", "kase", "loop_S", "loop_P", "k", "expr_sub", "N", "K",
                                          "needs_mask", "counter", "prd_engine", "cns_engine", "forward",
                                          "snap_slots")]


class StaticWait(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("dep", "same_region", "prd_engine", "ordinal")]


class Stats(C.Structure):
    _fields_ = [(n, C.c_int32) for n in ("n_counters", "regs_per_engine", "salu_ops_per_wait", "n_waits",
                                          "n_sync_points", "n_fallback")]


class RunOpts(C.Structure):
    _fields_ = [("watchdog_polls", C.c_uint64), ("fault_dep", C.c_int32), ("fault_delta", C.c_int32),
                ("dev_stats", C.c_void_p), ("k_unroll", C.c_int32), ("flags", C.c_uint32)]

RUN_PER_INSTANCE = 1
RUN_LOG_BATCHED = 2

STAT_FIELDS = ("run", "blocked", "n_blocked", "barrier", "own_loads", "polls")


_lib = None


def lib():
    """The loaded libbfs; raises if it was not built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"libbfs.so not built at {LIB_PATH}: run __graft_entry__.build()")
        L = C.CDLL(LIB_PATH)
        L.bfs_plan_create.restype = C.c_int
        L.bfs_plan_create.argtypes = [C.c_void_p, C.c_int, C.c_int, C.c_uint32, C.POINTER(C.c_void_p)]
        L.bfs_plan_formulas.restype = C.c_int
        L.bfs_plan_formulas.argtypes = [C.c_void_p, C.POINTER(C.POINTER(Formula)), C.POINTER(C.c_int32)]
        L.bfs_plan_static_waits.restype = C.c_int
        L.bfs_plan_static_waits.argtypes = [C.c_void_p, C.POINTER(C.POINTER(StaticWait)), C.POINTER(C.c_int32)]
        L.bfs_plan_stats.restype = C.c_int
        L.bfs_plan_stats.argtypes = [C.c_void_p, C.POINTER(Stats)]
        L.bfs_eval_threshold.restype = C.c_int
        L.bfs_eval_threshold.argtypes = [C.c_void_p, C.c_int32, C.c_uint32, C.c_uint32, C.POINTER(C.c_uint32)]
        L.bfs_plan_destroy.restype = None
        L.bfs_plan_destroy.argtypes = [C.c_void_p]
        L.bfs_run.restype = C.c_int
        L.bfs_run.argtypes = [C.c_void_p, C.c_void_p, C.c_int32, C.c_void_p, C.c_void_p, C.c_int32,
                              C.c_void_p, C.c_void_p, C.c_int64, C.c_void_p]
        L.bfs_run_noalloc.restype = C.c_int
        L.bfs_run_noalloc.argtypes = L.bfs_run.argtypes
        L.bfs_run_status.restype = C.c_int
        L.bfs_run_status.argtypes = [C.c_void_p, C.c_void_p]
        L.bfs_status_string.restype = C.c_char_p
        L.bfs_status_string.argtypes = [C.c_int]
        L.bfs_last_error.restype = C.c_char_p
        L.bfs_last_error.argtypes = []
        _lib = L
    return _lib


def _check(st):
    if st != OK:
        raise BfsError(st, lib().bfs_last_error().decode())


def _i32(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.int32))


def _ptr(x):
    """Device pointer of a torch tensor, or an int passed through."""
    if x is None:
        return None
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream_handle(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Plan:
    """A planned program (bfs_plan_create) with its owned C arrays."""

    def __init__(self, program, mode=MODE_BARRIER_FREE, alloc=ALLOC_PER_LOOP, fallback=False):
        """fallback: keep dependencies outside the allocatable cases and order
        them by barriers (BFS_PLAN_BARRIER_FALLBACK)."""
        f = program.flat() if hasattr(program, "flat") else program
        self._keep = [
            _i32(f["loop_parent"]), _i32(f["loop_is_cond"]), _i32(f["body_off"]), _i32(f["body_kind"] or [0]),
            _i32(f["body_id"] or [0]), _i32(f["block_off"]), _i32(f["block_instrs"] or [0]),
            _i32(f["instr_engine"] or [0]), _i32(f["instr_opcode"] or [0]),
            _i32(np.array(f["instr_args"] or [[0] * 8]).reshape(-1)),
            _i32(np.array(f["deps"] or [(0, 0, 0)]).reshape(-1)),
            _i32(f.get("dep_linear") or [0]),
        ]
        k = self._keep
        wpe = (C.c_int32 * 8)(*f["waves_per_engine"][:8])
        rs = (C.c_int32 * 4)(*f["ring_slots"][:4])
        kernel = f["kernel"] if isinstance(f["kernel"], int) else KERNELS[f["kernel"]]
        self._prog = _Program(kernel, f["n_engines"], wpe, len(f["loop_parent"]), k[0].ctypes.data,
                              k[1].ctypes.data, k[2].ctypes.data, k[3].ctypes.data, k[4].ctypes.data,
                              len(f["block_off"]) - 1, k[5].ctypes.data, k[6].ctypes.data,
                              len(f["instr_engine"]), k[7].ctypes.data, k[8].ctypes.data, k[9].ctypes.data,
                              len(f["deps"]), k[10].ctypes.data, f["tile_elems"], rs, f["n_accs"],
                              k[11].ctypes.data if f.get("dep_linear") else None)
        h = C.c_void_p()
        flags = PLAN_BARRIER_FALLBACK if fallback else 0
        _check(lib().bfs_plan_create(C.addressof(self._prog), mode, alloc, flags, C.byref(h)))
        self.handle = h
        self.mode = mode
        self.alloc = alloc
        self.n_loops = len(f["loop_parent"])
        self.n_engines = f["n_engines"]
        self.waves_per_engine = list(f["waves_per_engine"][: f["n_engines"]])

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value and _lib is not None:
            _lib.bfs_plan_destroy(h)
            self.handle = None

    @property
    def n_waves(self):
        return sum(self.waves_per_engine)

    def formulas(self):
        p = C.POINTER(Formula)()
        n = C.c_int32()
        _check(lib().bfs_plan_formulas(self.handle, C.byref(p), C.byref(n)))
        return [{k: getattr(p[i], k) for k, _ in Formula._fields_} for i in range(n.value)]

    def static_waits(self):
        p = C.POINTER(StaticWait)()
        n = C.c_int32()
        _check(lib().bfs_plan_static_waits(self.handle, C.byref(p), C.byref(n)))
        return [{k: getattr(p[i], k) for k, _ in StaticWait._fields_} for i in range(n.value)]

    def stats(self):
        s = Stats()
        _check(lib().bfs_plan_stats(self.handle, C.byref(s)))
        return {k: getattr(s, k) for k, _ in Stats._fields_}

    def eval_threshold(self, dep, r_P, rhat_S):
        out = C.c_uint32()
        _check(lib().bfs_eval_threshold(self.handle, dep, r_P, rhat_S, C.byref(out)))
        return out.value

    def run(self, buffers, trips, trip_off, n_wg, stream=None, debug_log=None, debug_capacity=0,
            watchdog_polls=0, fault_dep=-1, fault_delta=0, stats=None, k_unroll=0, flags=0):
        """Enqueue one execution (asynchronous).  buffers: torch tensors or
        device addresses; trips / trip_off: device int32 / int64 tensors;
        stats: optional int64 tensor of n_wg * n_waves * 8 per-wave counters;
        k_unroll: K-loop unroll factor of GEMM launches (0, 1, 2, 4, 8);
        flags: RUN_PER_INSTANCE / RUN_LOG_BATCHED (stream family)."""
        arr = (C.c_void_p * max(1, len(buffers)))(*[_ptr(b) for b in buffers])
        opts = RunOpts(watchdog_polls, fault_dep, fault_delta, _ptr(stats), k_unroll, flags)
        _check(lib().bfs_run(self.handle, arr, len(buffers), _ptr(trips), _ptr(trip_off), n_wg,
                             _stream_handle(stream), _ptr(debug_log), debug_capacity, C.byref(opts)))

    def run_noalloc(self, buffers, trips, trip_off, n_wg, stream=None, debug_log=None, debug_capacity=0,
                    watchdog_polls=0, fault_dep=-1, fault_delta=0, stats=None, k_unroll=0, flags=0):
        """As run(), through bfs_run_noalloc: the plan's tables and error words
        live in the library's fixed device array instead of an allocation."""
        arr = (C.c_void_p * max(1, len(buffers)))(*[_ptr(b) for b in buffers])
        opts = RunOpts(watchdog_polls, fault_dep, fault_delta, _ptr(stats), k_unroll, flags)
        _check(lib().bfs_run_noalloc(self.handle, arr, len(buffers), _ptr(trips), _ptr(trip_off), n_wg,
                                     _stream_handle(stream), _ptr(debug_log), debug_capacity, C.byref(opts)))

    def status(self, stream=None):
        """Synchronize the stream; raise BfsError(E_DEADLOCK) if a wait gave up."""
        _check(lib().bfs_run_status(self.handle, _stream_handle(stream)))

    def debug_log_words(self, n_wg, capacity):
        return n_wg * self.n_waves * (1 + 4 * capacity)


def parse_debug_log(words: np.ndarray, n_wg: int, n_waves: int, capacity: int):
    """Split a debug-log buffer into per-(workgroup, wave) entry arrays
    [n, 4] of (dependency, consumer instance, threshold, observed)."""
    words = np.asarray(words, dtype=np.uint32)
    counts = words[: n_wg * n_waves].reshape(n_wg, n_waves)
    ent = words[n_wg * n_waves:].reshape(n_wg, n_waves, capacity, 4)
    out = {}
    for w in range(n_wg):
        for v in range(n_waves):
            n = int(counts[w, v])
            if n > capacity:
                raise ValueError(f"debug log overflow in workgroup {w} wave {v}: {n} > {capacity}")
            out[(w, v)] = ent[w, v, :n].copy()
    return out
