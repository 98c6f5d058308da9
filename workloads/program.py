"""Structured loop programs: the input of the synchronization method.

A program is the statement tree of the paper's program model (Section 4.1 and
the grammar of Section 7.1): a top-level loop that runs once, whose body is a
sequence of blocks and nested loops.  A block lists datapath instructions in
one sequential program order; each instruction names the engine that runs it,
so an engine's instruction stream for the block is the projection of that
listing onto the engine (the block stream f of Appendix A.1).  A dependency is
the triple (producer, consumer, offset) of Appendix A.1 / Section 5.1.

This module only *describes* programs.  It holds none of the method's
arithmetic: no thresholds, no loop registers and no counters.  Both the CPU
oracle and the GPU library consume the description produced here.

Opcodes of the generic tile machine (the datapath semantics the instructions
carry, the instrOp of Appendix A.1).  A tile is ``tile_elems`` fp32 values.
Ring slots and global tile indices are addressed from loop-iteration counts:

* ``slot = ((r[gen_loop] - 1) % n_gen) * per_gen + ((rhat[pos_loop] - 1) % per_gen)``
  where ``r`` counts every iteration of a loop since the start of the
  workgroup and ``rhat`` counts iterations of the current trip; a ``gen_loop``
  of -1 drops the first term.
* ``gidx = base[wg] + r[idx_loop] - 1`` where ``base`` is the int64 per-workgroup
  tile base table (device buffer 0 for the tile-machine families).

Instruction argument layout ``args[8]``:
  0 src operand (ring id or buffer id), 1 dst operand (ring / buffer / acc id),
  2 gen_loop, 3 n_gen, 4 pos_loop, 5 per_gen, 6 idx_loop, 7 fp32 constant bits.
"""
from __future__ import annotations

import struct
from contextlib import contextmanager
from dataclasses import dataclass, field

# --- tile-machine opcodes -------------------------------------------------
OP_NOP = 0        # no datapath effect (an acquire / marker instruction)
OP_LOAD = 1       # ring[dst][slot] <- buffer[src] tile gidx
OP_SCALE_ACC = 2  # acc[dst] += const * ring[src][slot]
OP_STORE_ACC = 3  # buffer[dst] tile wg <- acc[src]
OP_ADDC = 4       # ring[dst][slot] <- ring[src][slot] + const
OP_STORE_RING = 5 # buffer[dst] tile gidx <- ring[src][slot]

# --- descriptive opcodes of the fused MFMA families (values are checked
# against the plain mathematical definition, not interpreted) --------------
OP_GEMM_LOAD = 16      # args: M, N, K (the shape of the whole product)
OP_GEMM_MMA = 17
OP_GEMM_SPILL = 18
OP_GEMM_EPI = 19
OP_GEMM_BIAS = 20      # stage the workgroup's bias columns in LDS
OP_ATTN_LOAD = 32
OP_ATTN_QK = 33
OP_ATTN_SM = 34
OP_ATTN_PV = 35
OP_ATTN_NORM = 36
OP_ATTN_PREAD = 37     # P fragments and alpha of the step into the PV waves' registers
OP_MOE_LOAD = 48       # args: phase (1 gate/up, 2 down), K, N, ring depth
OP_MOE_MMA = 49
OP_MOE_EPI = 50
OP_MOE_SPILL = 51      # args: epilogue ring depth
OP_RMS_LOAD = 64       # args: T, H, x-ring depth
OP_RMS_NORM = 65       # args: q-ring depth, eps (fp32 bits)
OP_RMS_STORE = 66
OP_ADAM_LOAD = 80      # args: N, chunk, ring depth
OP_ADAM_UPDATE = 81    # args: lr, beta1, beta2, eps, weight decay (fp32 bits), step t
OP_ADAM_STORE = 82

KIND_BLOCK = 0
KIND_LOOP = 1

KERNELS = ("interp", "stream3", "gemm", "attn", "moe", "rmsnorm", "adamw", "chain")


def f32_bits(x: float) -> int:
    """fp32 bit pattern of ``x`` as a signed int32 (instruction immediate)."""
    return struct.unpack("<i", struct.pack("<f", x))[0]


@dataclass
class Instr:
    engine: int
    opcode: int
    args: list
    name: str


@dataclass
class Program:
    kernel: str
    n_engines: int
    waves_per_engine: list
    loop_parent: list = field(default_factory=lambda: [-1])
    loop_is_cond: list = field(default_factory=lambda: [0])
    loop_names: list = field(default_factory=lambda: ["top"])
    body: list = field(default_factory=lambda: [[]])      # per loop: [(kind, id)]
    blocks: list = field(default_factory=list)             # per block: [instr id]
    instrs: list = field(default_factory=list)             # [Instr]
    deps: list = field(default_factory=list)               # [(prd, cns, k)]
    dep_linear: list = field(default_factory=list)         # per dep: 1 = linearized offset (extension), or empty
    tile_elems: int = 64
    ring_slots: list = field(default_factory=list)         # slots per ring
    n_accs: int = 0

    # ---- convenience lookups (pure structure, no method arithmetic) -----
    @property
    def n_loops(self) -> int:
        return len(self.loop_parent)

    def instr_id(self, name: str) -> int:
        for i, ins in enumerate(self.instrs):
            if ins.name == name:
                return i
        raise KeyError(name)

    def loop_id(self, name: str) -> int:
        return self.loop_names.index(name)

    def flat(self) -> dict:
        """Flat integer arrays (CSR) used by both the oracle and the library."""
        if any(self.dep_linear) and len(self.dep_linear) != len(self.deps):
            raise ValueError("dep_linear must have one flag per dependency")
        body_off, body = [0], []
        for items in self.body:
            body.extend(items)
            body_off.append(len(body))
        block_off, block_instrs = [0], []
        for b in self.blocks:
            block_instrs.extend(b)
            block_off.append(len(block_instrs))
        # block listings must enumerate instrs 0..n-1 in block order, so that
        # instruction ids double as sequential positions inside blocks.
        return dict(
            kernel=KERNELS.index(self.kernel),
            n_engines=self.n_engines,
            waves_per_engine=list(self.waves_per_engine) + [0] * (8 - len(self.waves_per_engine)),
            loop_parent=list(self.loop_parent),
            loop_is_cond=list(self.loop_is_cond),
            body_off=body_off,
            body_kind=[k for k, _ in body],
            body_id=[i for _, i in body],
            block_off=block_off,
            block_instrs=block_instrs,
            instr_engine=[ins.engine for ins in self.instrs],
            instr_opcode=[ins.opcode for ins in self.instrs],
            instr_args=[list(ins.args) + [0] * (8 - len(ins.args)) for ins in self.instrs],
            deps=[tuple(d) for d in self.deps],
            dep_linear=[int(x) for x in self.dep_linear] if any(self.dep_linear) else [],
            tile_elems=self.tile_elems,
            ring_slots=list(self.ring_slots) + [0] * (4 - len(self.ring_slots)),
            n_accs=self.n_accs,
        )


class ProgramBuilder:
    """Builds a Program with nested ``with b.loop(name):`` scopes.

    Instructions added consecutively without an intervening loop go into the
    same block, in the order they are added (the sequential listing)."""

    def __init__(self, kernel: str, n_engines: int, waves_per_engine=None):
        self.p = Program(kernel=kernel, n_engines=n_engines,
                         waves_per_engine=list(waves_per_engine or [1] * n_engines))
        self._stack = [0]
        self._open_block = {0: None}

    @contextmanager
    def loop(self, name: str, is_cond: bool = False):
        parent = self._stack[-1]
        lid = len(self.p.loop_parent)
        self.p.loop_parent.append(parent)
        self.p.loop_is_cond.append(1 if is_cond else 0)
        self.p.loop_names.append(name)
        self.p.body.append([])
        self.p.body[parent].append((KIND_LOOP, lid))
        self._open_block[parent] = None
        self._open_block[lid] = None
        self._stack.append(lid)
        try:
            yield lid
        finally:
            self._stack.pop()

    def block_break(self):
        """Start a new block in the current loop body at the next instruction."""
        self._open_block[self._stack[-1]] = None

    def instr(self, engine: int, opcode: int = OP_NOP, args=None, name=None) -> int:
        cur = self._stack[-1]
        if self._open_block.get(cur) is None:
            bid = len(self.p.blocks)
            self.p.blocks.append([])
            self.p.body[cur].append((KIND_BLOCK, bid))
            self._open_block[cur] = bid
        iid = len(self.p.instrs)
        self.p.instrs.append(Instr(engine, opcode, list(args or [0] * 8), name or f"i{iid}"))
        self.p.blocks[self._open_block[cur]].append(iid)
        return iid

    def dep(self, producer, consumer, offset: int, linear: bool = False):
        """``linear``: the offset counts iterations of the shared loop across
        its trips (an extension of the paper's relation; see the C header)."""
        if isinstance(producer, str):
            producer = self.p.instr_id(producer)
        if isinstance(consumer, str):
            consumer = self.p.instr_id(consumer)
        self.p.deps.append((producer, consumer, offset))
        self.p.dep_linear.append(1 if linear else 0)

    def build(self) -> Program:
        # Renumber instructions so that the concatenation of the blocks (in
        # block order) lists ids 0..n-1; deps are remapped accordingly.
        order = [i for b in self.p.blocks for i in b]
        remap = {old: new for new, old in enumerate(order)}
        self.p.instrs = [self.p.instrs[old] for old in order]
        self.p.blocks = [[remap[i] for i in b] for b in self.p.blocks]
        self.p.deps = [(remap[a], remap[b], k) for a, b, k in self.p.deps]
        return self.p


def tile_args(src=0, dst=0, gen_loop=-1, n_gen=1, pos_loop=-1, per_gen=1, idx_loop=-1, const=0.0):
    return [src, dst, gen_loop, n_gen, pos_loop, per_gen, idx_loop, f32_bits(const)]
