"""Loader for the paper-figure fixtures in tests/golden/."""
import glob
import json
import os

import numpy as np

from workloads import OP_NOP, ProgramBuilder, TripTables, draw_trips

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _emit(b, items):
    for it in items:
        if it[0] == "instr":
            b.instr(it[1], OP_NOP, name=it[2])
        else:
            with b.loop(it[1]):
                _emit(b, it[2])


def load(name):
    with open(os.path.join(GOLDEN, name)) as f:
        fx = json.load(f)
    b = ProgramBuilder("interp", fx["engines"])
    _emit(b, fx["program"])
    for p, c, k in fx["deps"]:
        b.dep(p, c, k)
    prog = b.build()

    def draw(l, n):
        t = np.asarray(fx["trips"][prog.loop_names[l]], dtype=np.int32)
        assert len(t) == n, (prog.loop_names[l], n, t)
        return t
    tt = TripTables([draw_trips(prog, draw)])
    return fx, prog, tt


def all_fixtures():
    return sorted(os.path.basename(p) for p in glob.glob(os.path.join(GOLDEN, "fig_*.json")))
