"""Paper arithmetic used to size and judge the path -- TEST INFRASTRUCTURE.

Closed forms written from the paper:
  * eq. (1): KV bytes per token 2*L*n_kv*d*p and per-layer chunk slice
    S = 2*G*n_kv*d*p;
  * eq. (2): size-threshold mode dispatch on W = N*L*S;
  * eq. (3): layerwise-prefetch TTFT  X_0 + sum_{l<L-1} max(X_{l+1}, C_l) + C_{L-1};
  * Section 3.5: the chunkwise baseline waits for all transfers first,
    sum X_l + sum C_l;
  * Section 5.3: overlap requirement B_req = D_l / t_l with
    D_l = 2*n_kv*d*p*(P*r);
  * Section 3.6, eq. (4): per-layer stall and the zero-stall rate r* = s/c;
  * Section 3.6, eqs. (5)-(7) and the evaluation's baselines: per-request
    bandwidth under a shared cap B -- Equal, KV-prop, BW-prop, Stall-opt and
    Calibrated Stall-opt;
  * Section 3.6, the scheduling-epoch rule: rates stay fixed while a
    request's KV loads, and a finished request's rate returns to the pool
    for the next epoch only.
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


def chunkwise_ttft(X: Sequence[float], C: Sequence[float]) -> float:
    """Section 3.5's chunkwise baseline: compute waits for the whole cached
    prefix, so every transfer comes before every layer's compute."""
    if len(X) != len(C) or not X:
        raise ValueError("X and C need one entry per layer")
    return float(sum(X)) + float(sum(C))


def required_bandwidth(context: int, hit: float, n_kv: int, d: int, t_layer_s: float,
                       p: int = 2) -> float:
    """Section 5.3: B_req = D_l / t_l in bytes/s, D_l = 2 n_kv d p (P r)."""
    return 2 * n_kv * d * p * (context * hit) / t_layer_s


def per_layer_stall(s: float, r: float, c: float) -> float:
    """eq. (4): max(0, s/r - c)."""
    return max(0.0, s / r - c)


def zero_stall_rate(s: float, c: float) -> float:
    return s / c


# ---------------------------------------------------------------------------
# bandwidth allocation under a shared cap (Section 3.6; the baselines of the
# multi-tenant evaluation).  s[i]: KV bytes request i transfers per layer;
# c[i]: its per-layer compute window in seconds; B: shared budget in bytes/s.
# ---------------------------------------------------------------------------

def alloc_equal(B: float, n: int):
    """Equal: the same share for every active request."""
    return [B / n] * n


def alloc_kv_prop(B: float, s: Sequence[float]):
    """KV-prop: shares proportional to the retrieved KV bytes (per layer
    bytes are the total over L, so the proportion is the same)."""
    tot = float(sum(s))
    return [B * x / tot for x in s]


def alloc_bw_prop(B: float, s: Sequence[float], c: Sequence[float]):
    """BW-prop: shares proportional to the zero-stall rates r*_i = s_i/c_i."""
    rs = [zero_stall_rate(a, b) for a, b in zip(s, c)]
    tot = sum(rs)
    return [B * x / tot for x in rs]


def stall_opt(B: float, s: Sequence[float], caps: Sequence[float]):
    """eq. (6): minimise sum_i s_i / r_i  s.t.  sum_i r_i = B, 0 < r_i <= cap_i.

    The objective is convex; at the optimum every request below its cap has
    the same marginal value s_i / r_i^2 = lambda, so r_i = min(cap_i,
    sqrt(s_i / lambda)).  sum_i r_i(lambda) falls as lambda grows: bisect on
    lambda until the budget is met.  When the caps fit in B every request
    gets its cap and the rest of the budget stays unassigned."""
    if sum(caps) <= B:
        return list(caps)

    def total(lam):
        return sum(min(cp, (x / lam) ** 0.5) for x, cp in zip(s, caps))

    lo, hi = 1e-300, 1.0
    while total(hi) > B:          # grow hi until the rates fit
        hi *= 4.0
    while total(lo) < B:          # lambda small enough that every request is capped
        lo /= 4.0
    for _ in range(400):
        mid = (lo * hi) ** 0.5
        if total(mid) > B:
            lo = mid
        else:
            hi = mid
        if hi / lo < 1 + 1e-15:
            break
    lam = (lo * hi) ** 0.5
    return [min(cp, (x / lam) ** 0.5) for x, cp in zip(s, caps)]


def alloc_stall_opt(B: float, s: Sequence[float], c: Sequence[float]):
    """Stall-opt (eqs. (5)-(6)): caps at the zero-stall rates."""
    return stall_opt(B, s, [zero_stall_rate(a, b) for a, b in zip(s, c)])


def alloc_cal_stall_opt(B: float, s: Sequence[float], c: Sequence[float], delta: float):
    """Calibrated Stall-opt (eq. (7)): the same program with the targets
    r*_i + delta as caps."""
    return stall_opt(B, s, [zero_stall_rate(a, b) + delta for a, b in zip(s, c)])


def total_stall(s: Sequence[float], c: Sequence[float], r: Sequence[float]) -> float:
    """Sum of the per-layer stalls of eq. (4)."""
    return sum(per_layer_stall(a, x, b) for a, b, x in zip(s, c, r))


# ---------------------------------------------------------------------------
# scheduling epochs (Section 3.6).  Requests arrive over time; in each
# scheduling epoch the requests that have arrived and are not yet served are
# admitted as one batch under the budget not held by requests still loading,
# with the batch's policy.  A request keeps its rate until its L layer
# payloads are delivered; the rate it frees goes back to the pool and is only
# handed out at a later epoch, never to a request already loading.  Reading
# taken where the paper gives no epoch length: with epoch > 0, epochs begin
# at the multiples of `epoch`; with epoch == 0, an epoch begins whenever a
# request arrives or finishes its delivery.
# ---------------------------------------------------------------------------

def epoch_schedule(policy: str, s: Sequence[float], c, L: int, arrival: Sequence[float], B: float,
                   delta: float = 0.0, epoch: float = 0.0):
    """(rates, admission times) of requests with per-layer bytes s[i],
    per-layer compute c[i] (the policies that use it), L layers and arrival
    times arrival[i], under budget B.  policy: equal, kv_prop, bw_prop,
    stall_opt or cal_stall_opt (margin delta)."""
    n = len(s)

    def allocate(budget, idx):
        ss = [s[i] for i in idx]
        cc = [c[i] for i in idx] if c is not None else None
        if policy == "equal":
            return alloc_equal(budget, len(idx))
        if policy == "kv_prop":
            return alloc_kv_prop(budget, ss)
        if policy == "bw_prop":
            return alloc_bw_prop(budget, ss, cc)
        if policy == "stall_opt":
            return alloc_stall_opt(budget, ss, cc)
        if policy == "cal_stall_opt":
            return alloc_cal_stall_opt(budget, ss, cc, delta)
        raise ValueError(policy)

    rate, admit = [None] * n, [None] * n

    def end(i):                       # when request i's last payload byte goes out
        return admit[i] + L * s[i] / rate[i]

    def epoch_start(t):               # the first epoch beginning at or after t
        if epoch == 0:
            return t
        k = -(-t // epoch)            # ceil
        while k * epoch < t:
            k += 1
        return k * epoch

    t = epoch_start(0.0)
    while any(a is None for a in admit):
        loading = [i for i in range(n) if admit[i] is not None and end(i) > t]
        free = B - sum(rate[i] for i in loading)
        batch = [i for i in range(n) if admit[i] is None and arrival[i] <= t]
        if batch and free > 1e-9 * B:
            for i, r in zip(batch, allocate(free, batch)):
                rate[i], admit[i] = r, t
        # the next epoch: after the next arrival or end of a delivery
        later = [arrival[i] for i in range(n) if admit[i] is None and arrival[i] > t]
        later += [end(i) for i in range(n) if admit[i] is not None and end(i) > t]
        if any(a is None for a in admit):
            if not later:
                raise RuntimeError("requests wait while nothing loads")
            t = epoch_start(min(later))
    return rate, admit
