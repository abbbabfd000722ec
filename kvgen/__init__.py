"""Seeded synthetic inputs for the layerwise prefix-KV path.

This module only draws random numbers and random structure.  It is the one
piece of code that both the CPU oracle and the GPU path consume, so it holds
none of the method's arithmetic: no KV layout decoding, no paging, no
attention.  Everything it returns is an input.

Random streams are Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel
random numbers: as easy as 1, 2, 3", SC'11) as shipped by numpy.  Each stream
is keyed by (seed, tensor kind, request, layer) through Philox's 128-bit key,
so any tensor of any layer of any request can be regenerated on its own.
Normal variates are numpy's float32 standard normal, rounded to bfloat16 with
round-to-nearest-even.  bfloat16 values are carried as uint16 bit patterns.

The five workload presets carry the shapes the paper evaluates: a Llama 3.1 8B
shape (32 layers, 32 query / 8 KV heads, head dim 128) at 4K and 64K cached
prefixes, a concurrent batch of that shape, a 70B shape, and a tiny case.
"""
from __future__ import annotations

import math
import threading
from dataclasses import dataclass, field, replace
from typing import List, Optional, Sequence

import numpy as np

# tensor kinds, folded into the Philox key
KIND_KV = 1        # chunk-object bytes (the cached prefix)
KIND_Q = 2         # suffix queries
KIND_KNEW = 3      # suffix keys
KIND_VNEW = 4      # suffix values
KIND_TABLE = 5     # block-table permutation
KIND_LENGTHS = 6   # batch prefix lengths
KIND_WEIGHT = 7    # rest-of-layer weights (req = which matrix)
KIND_ACT = 8       # rest-of-layer input activations


def _philox(seed: int, kind: int, req: int = 0, layer: int = 0) -> np.random.Generator:
    if not (0 <= req < (1 << 24) and 0 <= layer < (1 << 24) and 0 <= kind < (1 << 16)):
        raise ValueError("stream coordinates out of range")
    k1 = (kind << 48) | (req << 24) | layer
    return np.random.Generator(np.random.Philox(key=[seed & ((1 << 64) - 1), k1]))


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (round to nearest, ties to even); NaN stays NaN."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).copy()
    nan = (u & 0x7FFFFFFF) > 0x7F800000
    u += ((u >> 16) & 1) + np.uint32(0x7FFF)
    out = (u >> 16).astype(np.uint16)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def normal_bf16(seed: int, kind: int, req: int, layer: int, n: int) -> np.ndarray:
    """n i.i.d. N(0,1) values rounded to bfloat16, from stream (seed, kind, req, layer)."""
    g = _philox(seed, kind, req, layer)
    return f32_to_bf16_bits(g.standard_normal(n, dtype=np.float32))


# ---------------------------------------------------------------------------
# cached-prefix bytes
# ---------------------------------------------------------------------------

def chunk_layer_slices(seed: int, req: int, layer: int, n_chunks: int, slice_elems: int) -> np.ndarray:
    """Random bfloat16 contents of the layer-`layer` slice of every chunk object.

    Returns uint16 [n_chunks, slice_elems]; row j is the slice that chunk object
    j stores for that layer.  The values are i.i.d.; this function does not
    interpret them.
    """
    return normal_bf16(seed, KIND_KV, req, layer, n_chunks * slice_elems).reshape(n_chunks, slice_elems)


def chunk_objects(seed: int, req: int, num_layers: int, n_chunks: int, slice_elems: int,
                  threads: int = 8) -> np.ndarray:
    """The immutable chunk objects of one cached prefix, as an object store holds them.

    Returns uint16 [n_chunks, num_layers, slice_elems]: object j is row j, its
    num_layers slices stored back to back.  Layers are drawn in parallel threads
    (numpy releases the GIL while filling).
    """
    out = np.empty((n_chunks, num_layers, slice_elems), dtype=np.uint16)

    def work(layers):
        for l in layers:
            out[:, l, :] = chunk_layer_slices(seed, req, l, n_chunks, slice_elems)

    threads = max(1, min(threads, num_layers))
    parts = [list(range(num_layers))[i::threads] for i in range(threads)]
    ts = [threading.Thread(target=work, args=(p,)) for p in parts]
    for t in ts:
        t.start()
    for t in ts:
        t.join()
    return out


def suffix_tensor(seed: int, kind: int, req: int, layer: int, shape: Sequence[int]) -> np.ndarray:
    """Random bfloat16 suffix tensor (queries, new keys or new values) of a layer."""
    n = int(np.prod(shape))
    return normal_bf16(seed, kind, req, layer, n).reshape(tuple(shape))


# ---------------------------------------------------------------------------
# rest-of-layer weights
# ---------------------------------------------------------------------------

WEIGHT_NAMES = ("w_o", "w_gate_up", "w_down", "w_qkv")


def layer_weight(seed: int, which: int, layer: int, K: int, N: int) -> np.ndarray:
    """Random [K][N] bfloat16 weight matrix, entries N(0, 1/K), so a product
    with unit-variance inputs keeps unit variance.  `which` indexes
    WEIGHT_NAMES."""
    g = _philox(seed, KIND_WEIGHT, which, layer)
    x = g.standard_normal(K * N, dtype=np.float32) * np.float32(K ** -0.5)
    return f32_to_bf16_bits(x).reshape(K, N)


def layer_weight_shapes(H: int, F: int, n_qkv: int):
    """[K][N] of W_o, W_gate_up, W_down, W_qkv."""
    return ((H, H), (H, 2 * F), (F, H), (H, n_qkv))


# ---------------------------------------------------------------------------
# random structure: block tables and batch lengths
# ---------------------------------------------------------------------------

def fisher_yates(seed: int, req: int, n: int) -> np.ndarray:
    """Uniform random permutation of range(n) by the Fisher-Yates shuffle.

    Uses bounded integer draws from the keyed Philox stream, one per step,
    so the permutation depends only on (seed, req, n).
    """
    g = _philox(seed, KIND_TABLE, req, 0)
    perm = np.arange(n, dtype=np.int64)
    if n > 1:
        # j_i uniform in [0, i] for i = n-1 .. 1
        highs = np.arange(n - 1, 0, -1, dtype=np.int64)
        js = g.integers(0, highs + 1)
        for i, j in zip(highs.tolist(), js.tolist()):
            perm[i], perm[j] = perm[j], perm[i]
    return perm


def block_tables(seed: int, pages_needed: Sequence[int], pool_pages: int) -> List[np.ndarray]:
    """Distinct random pool pages for each request.

    A seeded permutation of the pool is dealt round-robin to the requests (one
    page per request per round, skipping requests that already hold what they
    need), so requests sharing a pool get interleaved pages.
    """
    total = int(sum(pages_needed))
    if total > pool_pages:
        raise ValueError("pool too small for the requested pages")
    perm = fisher_yates(seed, 0, pool_pages)
    tables = [[] for _ in pages_needed]
    pos = 0
    while pos < total:
        for r, need in enumerate(pages_needed):
            if len(tables[r]) < need:
                tables[r].append(int(perm[pos]))
                pos += 1
    return [np.asarray(t, dtype=np.int32) for t in tables]


def batch_prefix_lengths(seed: int, n_req: int, lo: int, hi: int, quantum: int) -> List[int]:
    """Log-uniform prefix lengths in [lo, hi], rounded down to whole chunks."""
    g = _philox(seed, KIND_LENGTHS, 0, 0)
    u = g.random(n_req)
    raw = np.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))
    return [max(quantum, int(quantum * math.floor(x / quantum))) for x in raw]


# ---------------------------------------------------------------------------
# workload presets
# ---------------------------------------------------------------------------

@dataclass
class Workload:
    name: str
    num_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    chunk_tokens: int
    prefix_tokens: List[int]          # per request
    suffix_tokens: List[int]          # per request
    pool_pages: int
    seed: int
    rate_bytes_per_s: float = 12.5e9  # 100 Gbps producer cap
    description: str = ""

    @property
    def n_requests(self) -> int:
        return len(self.prefix_tokens)

    def pages_needed(self, r: int) -> int:
        return -(-self.prefix_tokens[r] // self.page_size)

    def n_chunks(self, r: int) -> int:
        return self.prefix_tokens[r] // self.chunk_tokens

    @property
    def slice_elems(self) -> int:
        # elements of one chunk object's layer slice: K and V rows of G tokens
        return 2 * self.chunk_tokens * self.num_kv_heads * self.head_dim


def _single(name, seed, L, nq, nkv, d, tp, ts, pool_mult=4, pool_pages=None, desc=""):
    need = -(-tp // 16)
    return Workload(name=name, num_layers=L, num_q_heads=nq, num_kv_heads=nkv, head_dim=d,
                    page_size=16, chunk_tokens=16, prefix_tokens=[tp], suffix_tokens=[ts],
                    pool_pages=pool_pages if pool_pages is not None else pool_mult * need,
                    seed=seed, description=desc)


def workload(name: str, seed: Optional[int] = None) -> Workload:
    """Preset workloads (all G = page size = 16 tokens, bfloat16)."""
    if name == "tiny":
        return _single("tiny", seed or 1, 2, 4, 2, 64, 256, 32, pool_pages=64,
                       desc="2 layers, 4q/2kv, d64, 256-token prefix + 32-token suffix, 64-page pool")
    if name == "8b-4k":
        return _single("8b-4k", seed or 2, 32, 32, 8, 128, 4096, 128,
                       desc="Llama-3-8B shape, 4096-token prefix + 128-token suffix")
    if name == "8b-64k":
        return _single("8b-64k", seed or 3, 32, 32, 8, 128, 65536, 512,
                       desc="Llama-3-8B shape, 65536-token prefix + 512-token suffix")
    if name == "batch8":
        s = seed or 4
        tps = batch_prefix_lengths(s, 8, 4096, 32768, 16)
        need = sum(-(-t // 16) for t in tps)
        return Workload(name="batch8", num_layers=32, num_q_heads=32, num_kv_heads=8, head_dim=128,
                        page_size=16, chunk_tokens=16, prefix_tokens=tps, suffix_tokens=[256] * 8,
                        pool_pages=4 * need, seed=s,
                        description="8 requests, Llama-3-8B shape, log-uniform prefixes in [4096, 32768] + 256")
    if name == "70b-32k":
        return _single("70b-32k", seed or 5, 80, 64, 8, 128, 32768, 512,
                       desc="70B shape (80 layers, 64q/8kv, d128), 32768-token prefix + 512-token suffix")
    # one GPU's share of 8b-64k split eight ways: by KV head (each GPU holds
    # one KV head and its four query heads), or by prefix pages (each GPU
    # holds an eighth of the prefix; the one with the suffix does the most)
    if name == "8b-64k-tp8":
        return _single("8b-64k-tp8", seed or 3, 32, 4, 1, 128, 65536, 512,
                       desc="8b-64k, one of 8 KV-head shards: 4q/1kv, 65536-token prefix + 512-token suffix")
    if name == "8b-64k-cp8":
        return _single("8b-64k-cp8", seed or 3, 32, 32, 8, 128, 8192, 512,
                       desc="8b-64k, one of 8 prefix-page shards: 8192 prefix tokens + the 512-token suffix")
    raise KeyError(name)


WORKLOADS = ["tiny", "8b-4k", "8b-64k", "batch8", "70b-32k"]
SHARD_WORKLOADS = ["8b-64k-tp8", "8b-64k-cp8"]


def with_chunk_tokens(wl: Workload, G: int) -> Workload:
    """The same workload stored in chunks of G tokens (every prefix must be a
    whole number of them); the name gains a "-g<G>" suffix."""
    if any(t % G for t in wl.prefix_tokens):
        raise ValueError(f"prefix lengths {wl.prefix_tokens} are not multiples of G={G}")
    return replace(wl, name=f"{wl.name}-g{G}", chunk_tokens=G)


# ---------------------------------------------------------------------------
# the multi-tenant scheduler workloads (Section 5's bandwidth-allocation
# evaluation): requests are cells of the appendix table "Per-layer compute
# time and required transfer throughput" (Llama 3.1 8B on A100, L = 32,
# 4096 B per token per layer): (context, hit rate) -> cached tokens and the
# measured per-layer compute time in ms.  Workloads A and B hold the 16K and
# 64K cells at 50 % and 87.5 % under 80 and 50 Gbps caps; C adds the 32K
# cells under 50 Gbps.  `scale` divides cached tokens and compute windows
# alike, so every request keeps its transfer/compute ratio at the same caps.
# ---------------------------------------------------------------------------

SCHEDULER_CELLS = {
    (16384, 0.5): (8192, 29.87), (16384, 0.875): (14336, 8.80),
    (32768, 0.5): (16384, 80.91), (32768, 0.875): (28672, 23.85),
    (65536, 0.5): (32768, 271.02), (65536, 0.875): (57344, 75.75),
}
SCHEDULER_WORKLOADS = {
    "A": (10.0e9, [(16384, 0.5), (16384, 0.875), (65536, 0.5), (65536, 0.875)]),
    "B": (6.25e9, [(16384, 0.5), (16384, 0.875), (65536, 0.5), (65536, 0.875)]),
    "C": (6.25e9, [(16384, 0.5), (16384, 0.875), (32768, 0.5), (32768, 0.875), (65536, 0.5), (65536, 0.875)]),
}


def scheduler_workload(name: str, scale: int = 4, suffix: int = 128, seed: int = 6):
    """Workload `name` of the scheduler evaluation on the Llama-3-8B shape:
    (Workload, per-request compute window in seconds per layer, cap in bytes/s)."""
    cap, cells = SCHEDULER_WORKLOADS[name]
    tps = [SCHEDULER_CELLS[c][0] // scale for c in cells]
    windows = [SCHEDULER_CELLS[c][1] / scale / 1e3 for c in cells]
    need = sum(-(-t // 16) for t in tps)
    wl = Workload(name=f"sched-{name}", num_layers=32, num_q_heads=32, num_kv_heads=8, head_dim=128,
                  page_size=16, chunk_tokens=16, prefix_tokens=tps, suffix_tokens=[suffix] * len(tps),
                  pool_pages=4 * need, seed=seed, rate_bytes_per_s=cap,
                  description=f"scheduler workload {name}: cells {cells}, cached tokens and windows / {scale}")
    return wl, windows, cap
