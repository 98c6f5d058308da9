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


# ---- RMSNorm + FP8 quantization -------------------------------------------
E4M3_MAX = 448.0      # largest finite OCP FP8 E4M3 ("fn") value: 1.75 * 2^8


def e4m3fn_encode(v):
    """OCP FP8 E4M3 codes (1 sign, 4 exponent bits with bias 7, 3 mantissa
    bits; no infinities) of fp64 values with |v| <= 464, rounding to nearest
    with ties to even.  Normal numbers are (1 + m/8) * 2^(e-7) for exponent
    fields e = 1..15 (field 15 with mantissa 7 is NaN, so 448 is the
    largest); subnormals are m/8 * 2^-6."""
    v = np.asarray(v, np.float64)
    a = np.abs(v)
    if np.any(a > 464.0) or np.any(~np.isfinite(a)):
        raise ValueError("outside the E4M3 range handled here")
    code = np.zeros(a.shape, np.int64)
    sub = a < 2.0 ** -6
    # subnormal: a multiple of 2^-9, rounded half to even (8 * 2^-9 is the
    # smallest normal, whose code 8 is exactly the carried value)
    code[sub] = np.rint(a[sub] / 2.0 ** -9).astype(np.int64)
    n = ~sub
    e = np.floor(np.log2(a[n])).astype(np.int64)
    # guard the log2 rounding at exact powers of two
    e = np.where(2.0 ** e > a[n], e - 1, e)
    e = np.where(2.0 ** (e + 1) <= a[n], e + 1, e)
    m = np.rint((a[n] / 2.0 ** e - 1.0) * 8.0).astype(np.int64)
    carry = m == 8
    e = np.where(carry, e + 1, e)
    m = np.where(carry, 0, m)
    code[n] = ((e + 7) << 3) | m
    code = np.minimum(code, 0x7E)          # |v| in (448, 464) rounds to 448
    return (code | np.where(np.signbit(v), 0x80, 0)).astype(np.uint8)


def e4m3fn_decode(c):
    c = np.asarray(c, np.int64)
    s = np.where(c & 0x80, -1.0, 1.0)
    e, m = (c >> 3) & 0xF, c & 7
    mag = np.where(e == 0, m / 8.0 * 2.0 ** -6, (1.0 + m / 8.0) * 2.0 ** (e - 7.0))
    return s * mag


def rmsnorm_fp8_rows(x_bits, g_bits, eps, rows):
    """RMSNorm followed by per-row dynamic FP8 quantization, for the given
    rows: y = x / sqrt(mean(x^2) + eps) * gamma; scale s = max|y| / 448
    (1 for an all-zero row); codes = E4M3(y / s).  Returns (codes uint8
    [n, H], scales fp64 [n], y / s fp64 [n, H])."""
    g = bf16_to_f32(g_bits).astype(np.float64)
    codes, scales, ts = [], [], []
    for r in rows:
        x = bf16_to_f32(x_bits[r]).astype(np.float64)
        y = x / np.sqrt(np.mean(x * x) + eps) * g
        amax = np.max(np.abs(y))
        s = amax / E4M3_MAX if amax > 0 else 1.0
        t = y / s
        codes.append(e4m3fn_encode(t))
        scales.append(s)
        ts.append(t)
    return np.array(codes), np.array(scales), np.array(ts)


def e4m3fn_ambiguous(t, rel=2.0 ** -18):
    """True where t lies within a relative ``rel`` of a rounding midpoint
    between two adjacent E4M3 values: there the code depends on the last
    bits of the fp32 arithmetic that produced t, and either neighbour is a
    correct rounding of the exact value."""
    t = np.asarray(t, np.float64)
    lo = e4m3fn_encode(t * (1.0 - rel))
    hi = e4m3fn_encode(t * (1.0 + rel))
    return lo != hi


# ---- AdamW ------------------------------------------------------------------
def adamw_step(p, g, m, v, lr, b1, b2, eps, wd, t):
    """One AdamW step (Adam with decoupled weight decay) in fp64:
    m' = b1 m + (1 - b1) g, v' = b2 v + (1 - b2) g^2, bias-corrected
    mhat = m' / (1 - b1^t), vhat = v' / (1 - b2^t), and
    p' = p - lr (mhat / (sqrt(vhat) + eps) + wd p).  Returns (p', m', v')."""
    p, g, m, v = (np.asarray(a, np.float64) for a in (p, g, m, v))
    m1 = b1 * m + (1.0 - b1) * g
    v1 = b2 * v + (1.0 - b2) * g * g
    mhat = m1 / (1.0 - b1 ** t)
    vhat = v1 / (1.0 - b2 ** t)
    return p - lr * (mhat / (np.sqrt(vhat) + eps) + wd * p), m1, v1
