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
    """Round float64 values to the nearest bfloat16, ties to even, in one
    rounding step.

    bfloat16 keeps 8 significant bits and float32's exponent range: a value
    in [2^(e-1), 2^e) has the spacing 2^(e-8) when e-1 >= -126 (normal), and
    below 2^-126 the fixed subnormal spacing 2^-133.  x divided by that
    spacing is exact in float64 (a power-of-two scale), rint rounds the
    quotient to the nearest integer with ties to even, and the product with
    the spacing is then a bfloat16 value (or 2^128, which is infinity).
    That value is exact in float32, whose upper 16 bits are the result."""
    x = np.asarray(x, dtype=np.float64)
    finite = np.isfinite(x)
    xf = np.where(finite, x, 0.0)
    _, e = np.frexp(xf)                              # |x| in [2^(e-1), 2^e)
    ulp = np.ldexp(1.0, np.maximum(e, -125) - 8)
    r = np.rint(xf / ulp) * ulp                      # the one rounding
    r = np.where(np.abs(r) >= 2.0 ** 128, np.copysign(np.inf, xf), r)
    r = np.where(finite, r, x)                       # infinities and NaN pass through
    with np.errstate(over="ignore"):
        f = r.astype(np.float32)                     # exact: r is a bfloat16 value
    out = (f.view(np.uint32) >> 16).astype(np.uint16)
    out[np.isnan(x)] = 0x7FC0
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
