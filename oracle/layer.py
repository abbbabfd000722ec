"""Rest-of-layer compute around the attention -- TEST INFRASTRUCTURE.

The compute window C_l of eq. (3) is what the miss tokens cost per layer
(Section 3.5); besides the attention every layer runs the same projections
and feed-forward network (Section 3.6, the footnote on per-layer windows).
This is that chain for a Llama-style layer, in float64 with the products
rounded to bfloat16 (nearest even) where a bfloat16 pipeline stores them:

    o    = A . W_o                      A: attention output [T][H], H = n_q*d
    gu   = o . W_gu                     [T][2F]: gate columns, then up columns
    act  = silu(gate) * up              silu(x) = x / (1 + e^-x)
    h    = act . W_down                 [T][H]
    qkv  = h . W_qkv                    [T][(n_q + 2 n_kv) d], the next layer's projection

Weights are [K][N] row-major (input features by output features).  Norms,
residuals and biases are left out: the window's cost is its GEMMs.
Matrices are numpy uint16 arrays of bfloat16 bit patterns.
"""
from __future__ import annotations

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def f64_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16, ties to even (via float32, whose own
    rounding is nearest even; the two roundings agree except on values
    within 2^-24 relative of a bfloat16 tie)."""
    f = np.asarray(x, dtype=np.float64).astype(np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    nan = np.isnan(f)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    out = r.astype(np.uint16)
    out[nan] = 0x7FC0
    return out


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def rest_of_layer(attn_out, w_o, w_gu, w_down, w_qkv):
    """The chain above; every stage as bfloat16 bits: dict o, gu, act, h, qkv."""
    A = bf16_to_f64(attn_out)
    o = f64_to_bf16(A @ bf16_to_f64(w_o))
    gu = f64_to_bf16(bf16_to_f64(o) @ bf16_to_f64(w_gu))
    F = gu.shape[1] // 2
    g, u = bf16_to_f64(gu[:, :F]), bf16_to_f64(gu[:, F:])
    act = f64_to_bf16(silu(g) * u)
    h = f64_to_bf16(bf16_to_f64(act) @ bf16_to_f64(w_down))
    qkv = f64_to_bf16(bf16_to_f64(h) @ bf16_to_f64(w_qkv))
    return {"o": o, "gu": gu, "act": act, "h": h, "qkv": qkv}


def gemm_flops(tokens: int, H: int, F: int, n_qkv: int) -> int:
    """Multiply-adds x 2 of the chain: O (H x H), gate+up (H x 2F), down
    (F x H) and QKV (H x n_qkv) on `tokens` rows."""
    return 2 * tokens * (H * H + H * 2 * F + F * H + H * n_qkv)
