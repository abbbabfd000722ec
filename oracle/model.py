"""Paper arithmetic used to size and judge the path -- TEST INFRASTRUCTURE.

Closed forms written from the paper:
  * eq. (1): KV bytes per token 2*L*n_kv*d*p and per-layer chunk slice
    S = 2*G*n_kv*d*p;
  * eq. (2): size-threshold mode dispatch on W = N*L*S;
  * eq. (3): layerwise-prefetch TTFT  X_0 + sum_{l<L-1} max(X_{l+1}, C_l) + C_{L-1};
  * Section 5.3: overlap requirement B_req = D_l / t_l with
    D_l = 2*n_kv*d*p*(P*r);
  * Section 3.6, eq. (4): per-layer stall and the zero-stall rate r* = s/c.
"""
from __future__ import annotations

from typing import Sequence


def kv_bytes_per_token(L: int, n_kv: int, d: int, p: int = 2) -> int:
    """eq. (1), left: bytes of K and V for one token over all layers."""
    return 2 * L * n_kv * d * p


def layer_chunk_bytes(G: int, n_kv: int, d: int, p: int = 2) -> int:
    """eq. (1), right: bytes of one layer of one G-token chunk (S)."""
    return 2 * G * n_kv * d * p


def layer_range(layer: int, S: int):
    """Byte range of layer `layer` inside a chunk object (Section 3.2)."""
    return layer * S, (layer + 1) * S


def mode_dispatch(n_chunks: int, L: int, S: int, theta: float) -> str:
    """eq. (2): chunkwise below the threshold, layerwise + aggregation at or above it."""
    W = n_chunks * L * S
    return "chunkwise" if W < theta else "layerwise"


def layerwise_ttft(X: Sequence[float], C: Sequence[float]) -> float:
    """eq. (3) with one-layer prefetch."""
    L = len(X)
    if L != len(C) or L == 0:
        raise ValueError("X and C need one entry per layer")
    t = X[0]
    for l in range(L - 1):
        t += max(X[l + 1], C[l])
    return t + C[L - 1]


def required_bandwidth(context: int, hit: float, n_kv: int, d: int, t_layer_s: float,
                       p: int = 2) -> float:
    """Section 5.3: B_req = D_l / t_l in bytes/s, D_l = 2 n_kv d p (P r)."""
    return 2 * n_kv * d * p * (context * hit) / t_layer_s


def per_layer_stall(s: float, r: float, c: float) -> float:
    """eq. (4): max(0, s/r - c)."""
    return max(0.0, s / r - c)


def zero_stall_rate(s: float, c: float) -> float:
    return s / c
