"""Plain fp64 definitions of the fused MFMA workloads.

TEST INFRASTRUCTURE ONLY.

Each loop program of the GEMM, attention and MoE families partitions one
contraction among its engines, so the values it must produce are the plain
mathematical definitions below (evaluated in fp64 from the bf16-exact inputs).
The sampled variants evaluate single output elements / rows one by one, which
is how full-size outputs are checked.
"""
from __future__ import annotations

import numpy as np
from scipy.special import erf

from workloads.tensors import bf16_to_f32


def gelu(x):
    """GELU with the exact Gauss error function: x * Phi(x)."""
    return 0.5 * x * (1.0 + erf(x / np.sqrt(2.0)))


def silu(x):
    return x / (1.0 + np.exp(-x))


# ---- GEMM + bias + GELU ---------------------------------------------------
def gemm_bias_gelu(a_bits, bt_bits, bias):
    a = bf16_to_f32(a_bits).astype(np.float64)
    bt = bf16_to_f32(bt_bits).astype(np.float64)
    return gelu(a @ bt.T + np.asarray(bias, np.float64)[None, :])


def gemm_bias_gelu_at(a_bits, bt_bits, bias, rows, cols):
    """Output elements (rows[i], cols[i]) one by one."""
    rows = np.asarray(rows)
    cols = np.asarray(cols)
    a = bf16_to_f32(a_bits[rows]).astype(np.float64)
    bt = bf16_to_f32(bt_bits[cols]).astype(np.float64)
    return gelu(np.einsum("ik,ik->i", a, bt) + np.asarray(bias, np.float64)[cols])


# ---- variable-length attention -------------------------------------------
def attention_rows(q_bits, k_bits, v_bits, cu_seqlens, scale, items):
    """Softmax attention output rows.  ``items`` = [(b, h, i)]: query row i of
    sequence b, head h attends to all keys of sequence b (no causal mask)."""
    out = []
    for b, h, i in items:
        s0, s1 = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        q = bf16_to_f32(q_bits[s0 + i, h]).astype(np.float64)
        k = bf16_to_f32(k_bits[s0:s1, h]).astype(np.float64)
        v = bf16_to_f32(v_bits[s0:s1, h]).astype(np.float64)
        s = (k @ q) * scale
        p = np.exp(s - s.max())
        out.append((p / p.sum()) @ v)
    return np.array(out)


def attention(q_bits, k_bits, v_bits, cu_seqlens, scale):
    """Full output [T, H, D] (small sizes)."""
    t, hh, d = q_bits.shape
    out = np.zeros((t, hh, d))
    for b in range(len(cu_seqlens) - 1):
        s0, s1 = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        for h in range(hh):
            q = bf16_to_f32(q_bits[s0:s1, h]).astype(np.float64)
            k = bf16_to_f32(k_bits[s0:s1, h]).astype(np.float64)
            v = bf16_to_f32(v_bits[s0:s1, h]).astype(np.float64)
            s = (q @ k.T) * scale
            p = np.exp(s - s.max(axis=1, keepdims=True))
            out[s0:s1, h] = (p / p.sum(axis=1, keepdims=True)) @ v
    return out


# ---- MoE: top-1 routed SiLU-gated MLP -------------------------------------
def moe_hidden(moe, tokens, weights=None):
    """The gated hidden rows h[t] = SiLU(x W_gate) * (x W_up) of the given
    tokens under their routed expert (the first half of the expert MLP)."""
    weights = weights if weights is not None else {}
    out = []
    for t in tokens:
        e = int(moe.assign[t])
        if e not in weights:
            weights[e] = tuple(bf16_to_f32(w).astype(np.float64) for w in moe.weights(e))
        wg, wu, _ = weights[e]
        x = bf16_to_f32(moe.x[t]).astype(np.float64)
        out.append(silu(wg @ x) * (wu @ x))
    return np.array(out)


def moe_tokens(moe, tokens, weights=None):
    """Outputs y[t] = (SiLU(x W_gate) * (x W_up)) W_down for the given tokens,
    using each token's routed expert (gate weight 1)."""
    weights = weights if weights is not None else {}
    out = []
    for t in tokens:
        e = int(moe.assign[t])
        if e not in weights:
            weights[e] = tuple(bf16_to_f32(w).astype(np.float64) for w in moe.weights(e))
        wg, wu, wd = weights[e]
        x = bf16_to_f32(moe.x[t]).astype(np.float64)
        h = silu(wg @ x) * (wu @ x)
        out.append(wd @ h)
    return np.array(out)
