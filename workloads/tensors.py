"""Seeded tensors for the fused MFMA workloads (GEMM, attention, MoE).

bf16 tensors are drawn in fp32 and rounded to nearest-even bf16; both sides
consume the rounded values (held here as uint16 bit patterns).
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np

from .configs import CFG_ADAM, CFG_ATTN, CFG_GEMM, CFG_MOE, CFG_RMS, rng_for


def to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 to nearest-even bf16, returned as uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> 16) & 1
    r = (u + np.uint32(0x7FFF) + lsb) >> 16
    return r.astype(np.uint16)


def bf16_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


# ---------------------------------------------------------------------------
# GEMM + bias + GELU
# ---------------------------------------------------------------------------
@dataclass
class GemmInputs:
    a: np.ndarray      # uint16 bf16 [M, K] row-major
    bt: np.ndarray     # uint16 bf16 [N, K]: column n of B stored contiguously in k
    bias: np.ndarray   # fp32 [N], added to every row (one value per output column)


def gemm_inputs(seed: int = 0, m: int = 4096, n: int = 4096, k: int = 4096) -> GemmInputs:
    g = rng_for(CFG_GEMM, seed, 0)
    a = to_bf16_bits(g.standard_normal((m, k), dtype=np.float32) / 64.0)
    bt = to_bf16_bits(rng_for(CFG_GEMM, seed, 1).standard_normal((n, k), dtype=np.float32) / 64.0)
    bias = rng_for(CFG_GEMM, seed, 2).standard_normal(n, dtype=np.float32)
    return GemmInputs(a, bt, bias)


# ---------------------------------------------------------------------------
# variable-length attention forward
# ---------------------------------------------------------------------------
@dataclass
class AttnInputs:
    q: np.ndarray          # uint16 bf16 [T, H, D] packed sequences
    k: np.ndarray
    v: np.ndarray
    cu_seqlens: np.ndarray # int32 [B + 1]
    lengths: np.ndarray    # int32 [B]


def attn_lengths(seed: int = 0, batch: int = 32, lmin: int = 128, lmax: int = 4096) -> np.ndarray:
    return rng_for(CFG_ATTN, seed, 0).integers(lmin, lmax + 1, size=batch).astype(np.int32)


def attn_inputs(seed: int = 0, batch: int = 32, heads: int = 16, dim: int = 128,
                lmin: int = 128, lmax: int = 4096, lengths=None) -> AttnInputs:
    lens = np.asarray(lengths, dtype=np.int32) if lengths is not None else attn_lengths(seed, batch, lmin, lmax)
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    t = int(cu[-1])
    out = []
    for i in range(3):
        g = rng_for(CFG_ATTN, seed, 1 + i)
        out.append(to_bf16_bits(g.standard_normal((t, heads, dim), dtype=np.float32)))
    return AttnInputs(out[0], out[1], out[2], cu, lens)


# ---------------------------------------------------------------------------
# MoE grouped GEMM (top-1, Zipf expert counts, SiLU-gated MLP)
# ---------------------------------------------------------------------------
def zipf_counts(tokens: int, experts: int, s: float = 1.1) -> np.ndarray:
    """Counts proportional to rank^-s, rounded by largest remainder to sum to
    ``tokens`` (rank 1 first)."""
    w = np.arange(1, experts + 1, dtype=np.float64) ** (-s)
    exact = tokens * w / w.sum()
    c = np.floor(exact).astype(np.int64)
    rem = tokens - int(c.sum())
    order = np.argsort(-(exact - c), kind="stable")
    c[order[:rem]] += 1
    return c


@dataclass
class MoeInputs:
    x: np.ndarray            # uint16 bf16 [T, hidden]
    assign: np.ndarray       # int32 [T]: expert of each token (top-1, gate weight 1)
    counts: np.ndarray       # int64 [E]
    perm: np.ndarray         # int32 [T]: token ids grouped by expert, ascending inside a group
    expert_off: np.ndarray   # int32 [E + 1]: group boundaries in perm
    hidden: int
    ffn: int
    seed: int

    def weights(self, e: int):
        """Expert e's weights as uint16 bf16: w_gate_t, w_up_t [ffn, hidden]
        (each output column contiguous in the hidden dim) and w_down_t
        [hidden, ffn] (each output column contiguous in the ffn dim)."""
        g = rng_for(CFG_MOE, self.seed, 1000 + e)
        wg = to_bf16_bits(g.standard_normal((self.ffn, self.hidden), dtype=np.float32) * 0.02)
        wu = to_bf16_bits(g.standard_normal((self.ffn, self.hidden), dtype=np.float32) * 0.02)
        wd = to_bf16_bits(g.standard_normal((self.hidden, self.ffn), dtype=np.float32) * 0.02)
        return wg, wu, wd


def moe_inputs(seed: int = 0, tokens: int = 32768, experts: int = 64, hidden: int = 4096,
               ffn: int = 1408, s: float = 1.1, counts=None) -> MoeInputs:
    """Top-1 routing with Zipf(s) expert counts over a seeded rank -> expert
    map (or the given per-expert ``counts``), a seeded shuffle of the token ->
    expert assignment, and x ~ N(0, 1) rounded to bf16."""
    g = rng_for(CFG_MOE, seed, 0)
    if counts is None:
        counts_by_rank = zipf_counts(tokens, experts, s)
        rank_to_expert = g.permutation(experts)
        counts = np.zeros(experts, np.int64)
        counts[rank_to_expert] = counts_by_rank
    else:
        counts = np.asarray(counts, np.int64)
        experts, tokens = len(counts), int(counts.sum())
    assign = np.repeat(np.arange(experts, dtype=np.int32), counts)
    g.shuffle(assign)
    perm = np.argsort(assign, kind="stable").astype(np.int32)
    expert_off = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    x = to_bf16_bits(rng_for(CFG_MOE, seed, 1).standard_normal((tokens, hidden), dtype=np.float32))
    return MoeInputs(x, assign, counts, perm, expert_off, hidden, ffn, seed)


def moe_weights_all(moe: MoeInputs):
    """Every expert's weights stacked: W_gate, W_up [E][ffn][hidden] and
    W_down [E][hidden][ffn], uint16 bf16."""
    E = len(moe.counts)
    wg = np.empty((E, moe.ffn, moe.hidden), np.uint16)
    wu = np.empty((E, moe.ffn, moe.hidden), np.uint16)
    wd = np.empty((E, moe.hidden, moe.ffn), np.uint16)
    for e in range(E):
        wg[e], wu[e], wd[e] = moe.weights(e)
    return wg, wu, wd


# ---------------------------------------------------------------------------
# RMSNorm + FP8 quantization
# ---------------------------------------------------------------------------
@dataclass
class RmsInputs:
    x: np.ndarray       # uint16 bf16 [T, H]
    gamma: np.ndarray   # uint16 bf16 [H]
    outliers: np.ndarray  # the channels drawn with a larger scale


def rmsnorm_inputs(seed: int = 0, t: int = 32768, h: int = 8192, outlier_frac: float = 0.005,
                   outlier_scale: float = 20.0) -> RmsInputs:
    """Activations x ~ N(0, 1) with a seeded 0.5 % of channels scaled by 20
    (the outlier channels that make per-row dynamic FP8 scaling matter), and
    gamma = 1 + N(0, 0.1) per channel; both rounded to bf16."""
    g = rng_for(CFG_RMS, seed, 0)
    n_out = max(1, int(round(outlier_frac * h)))
    outliers = np.sort(g.choice(h, size=n_out, replace=False))
    colscale = np.ones(h, np.float32)
    colscale[outliers] = outlier_scale
    gx = rng_for(CFG_RMS, seed, 1)
    x = np.empty((t, h), np.uint16)
    for r0 in range(0, t, 4096):
        r1 = min(t, r0 + 4096)
        x[r0:r1] = to_bf16_bits(gx.standard_normal((r1 - r0, h), dtype=np.float32) * colscale[None, :])
    gamma = to_bf16_bits(1.0 + 0.1 * rng_for(CFG_RMS, seed, 2).standard_normal(h, dtype=np.float32))
    return RmsInputs(x, gamma, outliers)


# ---------------------------------------------------------------------------
# AdamW
# ---------------------------------------------------------------------------
@dataclass
class AdamInputs:
    p: np.ndarray     # fp32 [N] parameters
    g: np.ndarray     # fp32 [N] gradients
    m: np.ndarray     # fp32 [N] first moments
    v: np.ndarray     # fp32 [N] second moments (>= 0)


def adamw_inputs(seed: int = 0, n: int = 1 << 20) -> AdamInputs:
    """Optimizer state of a model a few steps into training: p ~ N(0, 0.02),
    g ~ N(0, 0.01) with 1 % of entries 30x larger, m ~ N(0, 0.003),
    v = (N(0, 0.01))^2; all fp32."""
    g_ = rng_for(CFG_ADAM, seed, 0)
    p = (0.02 * g_.standard_normal(n)).astype(np.float32)
    g = 0.01 * g_.standard_normal(n)
    g[g_.random(n) < 0.01] *= 30.0
    m = (0.003 * g_.standard_normal(n)).astype(np.float32)
    v = ((0.01 * g_.standard_normal(n)) ** 2).astype(np.float32)
    return AdamInputs(p, g.astype(np.float32), m, v)
