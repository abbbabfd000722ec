"""ctypes binding of ``libobjectcache.so`` -- argument marshalling only.

Every function here has the name of the C entry point it calls and does no
arithmetic of the method: it turns torch tensors (device memory owned by the
caller) and Python ints into the C structs of ``include/objectcache.h`` and
raises ``OcError`` on a non-zero status.  The library must have been built
(``python -m paper_2605_22850_amd.build``); there is no fallback.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_double, c_int, c_int32, c_int64, c_size_t, c_void_p
from dataclasses import dataclass
from typing import Optional, Sequence

_HERE = os.path.dirname(os.path.abspath(__file__))
# OC_LIBRARY names another build of the same library (the sanitizer build of
# its host code, say); by default the in-tree one
LIB_PATH = os.environ.get("OC_LIBRARY") or os.path.join(_HERE, "libobjectcache.so")

OC_OK, OC_EINVAL, OC_ESHAPE, OC_EALIGN, OC_ERANGE, OC_EHIP, OC_ETIMEOUT, OC_ENOMEM, OC_EABORT, OC_ESHORT = \
    0, -1, -2, -3, -4, -5, -6, -7, -8, -9
OC_MODE_HBM_RESIDENT, OC_MODE_DEVICE_STAGED, OC_MODE_PRODUCER = 0, 1, 2
OC_FAULT_NONE, OC_FAULT_STALL, OC_FAULT_ABORT, OC_FAULT_SHORT_WRITE = 0, 1, 2, 3
ALLOC_POLICIES = {"fifo": 0, "equal": 1, "kv_prop": 2, "bw_prop": 3, "stall_opt": 4, "cal_stall_opt": 5}
DELIVERIES = {"layerwise": 0, "chunkwise": 1, "auto": 2}

EXPORTS = [
    "oc_abi_version", "oc_last_error", "oc_block_table_check", "oc_kv_layer_ingest", "oc_kv_chunks_ingest",
    "oc_kv_layer_gather", "oc_kv_chunks_gather", "oc_kv_suffix_append", "oc_rest_of_layer",
    "oc_attention_workspace_bytes", "oc_suffix_prefill_layer", "oc_context_create", "oc_pipeline_run",
    "oc_pipeline_last_ms", "oc_context_destroy", "oc_bandwidth_allocate", "oc_suffix_prefill_layer_noalloc",
    "oc_epoch_schedule",
]
OC_NOALLOC_WORKSPACE_BYTES = 65 << 20


class OcError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"objectcache status {status}: {msg}")
        self.status = status


class c_layout(ctypes.Structure):
    _fields_ = [("num_layers", c_int32), ("num_q_heads", c_int32), ("num_kv_heads", c_int32),
                ("head_dim", c_int32), ("page_size", c_int32), ("chunk_tokens", c_int32),
                ("num_pages", c_int64)]


class c_kv_pool(ctypes.Structure):
    _fields_ = [("base", c_void_p), ("layout", c_layout)]


class c_block_table(ctypes.Structure):
    _fields_ = [("pages", c_void_p), ("num_entries", c_int64), ("num_tokens", c_int64)]


class c_staging(ctypes.Structure):
    _fields_ = [("data", c_void_p), ("num_chunks", c_int64), ("per_layer_chunk_bytes", c_int64)]


class c_pipeline_opts(ctypes.Structure):
    _fields_ = [("mode", c_int32), ("rate_bytes_per_s", c_double), ("piece_bytes", c_int64),
                ("slots", c_int32), ("producer_threads", c_int32), ("timeout_ms", c_int32),
                ("fault", c_int32), ("fault_layer", c_int32), ("alloc_policy", c_int32),
                ("margin_bytes_per_s", c_double), ("delivery", c_int32), ("theta_bytes", c_double),
                ("emulate_compute", c_int32), ("append_suffix", c_int32), ("attention_per_request", c_int32),
                ("layer_weights", c_void_p), ("epoch_s", c_double)]


class c_layer_weights(ctypes.Structure):
    _fields_ = [("ffn_dim", c_int32), ("w_o", c_void_p), ("w_gate_up", c_void_p), ("w_down", c_void_p),
                ("w_qkv", c_void_p)]


class c_layer_buffers(ctypes.Structure):
    _fields_ = [("o", c_void_p), ("gate_up", c_void_p), ("act", c_void_p), ("h", c_void_p), ("qkv", c_void_p)]


class c_request(ctypes.Structure):
    _fields_ = [("prefix_tokens", c_int64), ("suffix_tokens", c_int64), ("block_table", POINTER(c_block_table)),
                ("chunk_objects", POINTER(c_void_p)), ("device_payload", c_void_p), ("q", c_void_p),
                ("k_new", c_void_p), ("v_new", c_void_p), ("out", c_void_p), ("layer_compute_s", c_double),
                ("arrival_s", c_double)]


class c_request_stats(ctypes.Structure):
    _fields_ = [("ttft_ms", c_double), ("produced_ms", POINTER(c_double)), ("landed_ms", POINTER(c_double)),
                ("ingested_ms", POINTER(c_double)), ("done_ms", POINTER(c_double)),
                ("rate_bytes_per_s", c_double), ("delivery", c_int32), ("admitted_ms", c_double)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2605_22850_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        L.oc_abi_version.restype = c_int
        L.oc_last_error.restype = ctypes.c_char_p
        L.oc_block_table_check.argtypes = [c_void_p, c_int64, c_int64, c_int64, c_int32]
        L.oc_kv_layer_ingest.argtypes = [POINTER(c_staging), POINTER(c_block_table), POINTER(c_kv_pool), c_int32,
                                         c_void_p]
        L.oc_kv_chunks_ingest.argtypes = [POINTER(c_staging), c_int64, POINTER(c_block_table), POINTER(c_kv_pool),
                                          c_void_p]
        L.oc_kv_layer_gather.argtypes = [POINTER(c_block_table), POINTER(c_kv_pool), c_int32, c_void_p, c_int64,
                                         c_int64, c_void_p]
        L.oc_kv_chunks_gather.argtypes = [POINTER(c_block_table), POINTER(c_kv_pool), c_int64, c_int64, c_void_p,
                                          c_void_p]
        L.oc_kv_suffix_append.argtypes = [c_void_p, c_void_p, c_int64, POINTER(c_block_table), POINTER(c_kv_pool),
                                          c_int32, c_void_p]
        L.oc_rest_of_layer.argtypes = [c_void_p, c_int64, POINTER(c_layout), POINTER(c_layer_weights), c_int32,
                                       POINTER(c_layer_buffers), c_void_p]
        L.oc_attention_workspace_bytes.argtypes = [POINTER(c_layout), c_int64, c_int64]
        L.oc_attention_workspace_bytes.restype = c_size_t
        L.oc_suffix_prefill_layer.argtypes = [c_void_p, c_void_p, c_void_p, c_int64, POINTER(c_kv_pool),
                                              POINTER(c_block_table), c_int32, c_void_p, c_void_p, c_size_t,
                                              c_void_p]
        L.oc_suffix_prefill_layer_noalloc.argtypes = [c_void_p, c_void_p, c_void_p, c_int64, POINTER(c_kv_pool),
                                                      POINTER(c_block_table), c_int32, c_void_p, c_void_p]
        if hasattr(L, "oc_pipeline_run"):
            L.oc_context_create.argtypes = [c_int, POINTER(c_kv_pool), POINTER(c_pipeline_opts), c_int64, c_int64,
                                            POINTER(c_void_p)]
            L.oc_context_create.restype = c_int
            L.oc_pipeline_run.argtypes = [c_void_p, POINTER(c_request), c_int32, POINTER(c_request_stats)]
            L.oc_pipeline_run.restype = c_int
            L.oc_pipeline_last_ms.argtypes = [c_void_p]
            L.oc_pipeline_last_ms.restype = c_double
            L.oc_context_destroy.argtypes = [c_void_p]
            L.oc_context_destroy.restype = None
        L.oc_bandwidth_allocate.argtypes = [c_int32, c_int32, POINTER(c_double), POINTER(c_double), c_double, c_double,
                                            POINTER(c_double)]
        L.oc_epoch_schedule.argtypes = [c_int32, c_int32, POINTER(c_double), POINTER(c_double), c_int32,
                                        POINTER(c_double), c_double, c_double, c_double, POINTER(c_double),
                                        POINTER(c_double)]
        for name in ("oc_block_table_check", "oc_kv_layer_ingest", "oc_kv_chunks_ingest", "oc_kv_layer_gather",
                     "oc_kv_chunks_gather", "oc_kv_suffix_append", "oc_rest_of_layer", "oc_suffix_prefill_layer",
                     "oc_suffix_prefill_layer_noalloc", "oc_bandwidth_allocate", "oc_epoch_schedule"):
            getattr(L, name).restype = c_int
        _lib = L
    return _lib


def _check(rc: int):
    if rc != OC_OK:
        raise OcError(rc, lib().oc_last_error().decode())


@dataclass
class Layout:
    num_layers: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    chunk_tokens: int
    num_pages: int

    def c(self) -> c_layout:
        return c_layout(self.num_layers, self.num_q_heads, self.num_kv_heads, self.head_dim, self.page_size,
                        self.chunk_tokens, self.num_pages)

    @property
    def slice_bytes(self) -> int:
        """S of eq. (1) with 2-byte elements."""
        return 2 * self.chunk_tokens * self.num_kv_heads * self.head_dim * 2

    @property
    def pool_elems(self) -> int:
        return self.num_layers * 2 * self.num_pages * self.num_kv_heads * self.page_size * self.head_dim


def _ptr(t) -> Optional[int]:
    if t is None:
        return None
    return t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def make_pool(pool, layout: Layout) -> c_kv_pool:
    return c_kv_pool(_ptr(pool), layout.c())


def make_table(pages, num_tokens: int) -> c_block_table:
    n = 0 if pages is None else pages.numel()
    return c_block_table(_ptr(pages) if n else None, n, num_tokens)


def oc_abi_version() -> int:
    return lib().oc_abi_version()


def oc_block_table_check(host_pages, num_tokens: int, num_pages: int, page_size: int) -> None:
    import numpy as np
    a = np.ascontiguousarray(host_pages, dtype=np.int32)
    _check(lib().oc_block_table_check(a.ctypes.data if a.size else None, a.size, num_tokens, num_pages, page_size))


def oc_kv_layer_ingest(staging, num_chunks: int, pages, num_tokens: int, pool, layout: Layout, layer: int,
                       stream=None) -> None:
    st = c_staging(_ptr(staging), num_chunks, layout.slice_bytes)
    bt = make_table(pages, num_tokens)
    kp = make_pool(pool, layout)
    _check(lib().oc_kv_layer_ingest(ctypes.byref(st), ctypes.byref(bt), ctypes.byref(kp), layer, _stream(stream)))


def oc_kv_chunks_ingest(objects, num_chunks: int, first_chunk: int, pages, num_tokens: int, pool, layout: Layout,
                        stream=None) -> None:
    """Whole chunk objects (device, num_chunks * L * S bytes back to back) -> every layer of the pool."""
    st = c_staging(_ptr(objects), num_chunks, layout.slice_bytes)
    bt = make_table(pages, num_tokens)
    kp = make_pool(pool, layout)
    _check(lib().oc_kv_chunks_ingest(ctypes.byref(st), first_chunk, ctypes.byref(bt), ctypes.byref(kp),
                                     _stream(stream)))


def oc_kv_layer_gather(pages, num_tokens: int, pool, layout: Layout, layer: int, staging_out, num_chunks: int,
                       stream=None) -> None:
    bt = make_table(pages, num_tokens)
    kp = make_pool(pool, layout)
    _check(lib().oc_kv_layer_gather(ctypes.byref(bt), ctypes.byref(kp), layer, _ptr(staging_out), num_chunks,
                                    layout.slice_bytes, _stream(stream)))


def oc_kv_chunks_gather(pages, num_tokens: int, pool, layout: Layout, first_chunk: int, num_chunks: int,
                        objects_out, stream=None) -> None:
    """Pool -> chunk objects first_chunk .. first_chunk+num_chunks-1 (all layers) into device objects_out."""
    bt = make_table(pages, num_tokens)
    kp = make_pool(pool, layout)
    _check(lib().oc_kv_chunks_gather(ctypes.byref(bt), ctypes.byref(kp), first_chunk, num_chunks,
                                     _ptr(objects_out), _stream(stream)))


def oc_kv_suffix_append(k_new, v_new, suffix_tokens: int, pages, num_tokens: int, pool, layout: Layout,
                        layer: int, stream=None) -> None:
    """One layer's suffix K/V (device [Ts][nkv][d]) -> pool positions num_tokens .. num_tokens+Ts-1."""
    bt = make_table(pages, num_tokens)
    kp = make_pool(pool, layout)
    _check(lib().oc_kv_suffix_append(_ptr(k_new), _ptr(v_new), suffix_tokens, ctypes.byref(bt), ctypes.byref(kp),
                                     layer, _stream(stream)))


@dataclass
class LayerWeights:
    """Device bf16 weights of the rest-of-layer window (torch tensors, [L][K][N]
    row-major each; the tensors must outlive every call or context using them)."""
    ffn_dim: int
    w_o: object             # [L][H][H], H = n_q * d
    w_gate_up: object       # [L][H][2F]
    w_down: object          # [L][F][H]
    w_qkv: object           # [L][H][(n_q + 2 n_kv) d]

    def c(self) -> c_layer_weights:
        return c_layer_weights(self.ffn_dim, _ptr(self.w_o), _ptr(self.w_gate_up), _ptr(self.w_down),
                               _ptr(self.w_qkv))


def oc_rest_of_layer(attn_out, tokens: int, layout: Layout, weights: LayerWeights, layer: int, o, gate_up, act, h,
                     qkv, stream=None) -> None:
    """The rest of one layer on `tokens` rows of attn_out; stage outputs into o, gate_up, act, h, qkv."""
    lay = layout.c()
    w = weights.c()
    b = c_layer_buffers(_ptr(o), _ptr(gate_up), _ptr(act), _ptr(h), _ptr(qkv))
    _check(lib().oc_rest_of_layer(_ptr(attn_out), tokens, ctypes.byref(lay), ctypes.byref(w), layer,
                                  ctypes.byref(b), _stream(stream)))


def oc_attention_workspace_bytes(layout: Layout, prefix_tokens: int, suffix_tokens: int) -> int:
    lay = layout.c()
    n = lib().oc_attention_workspace_bytes(ctypes.byref(lay), prefix_tokens, suffix_tokens)
    if n == 0:
        raise OcError(OC_EINVAL, lib().oc_last_error().decode() or "unsupported attention shape")
    return n


def oc_suffix_prefill_layer(q, k_new, v_new, suffix_tokens: int, pool, layout: Layout, pages, num_tokens: int,
                            layer: int, out, workspace, stream=None) -> None:
    bt = make_table(pages, num_tokens)
    kp = make_pool(pool, layout)
    _check(lib().oc_suffix_prefill_layer(_ptr(q), _ptr(k_new), _ptr(v_new), suffix_tokens, ctypes.byref(kp),
                                         ctypes.byref(bt), layer, _ptr(out), _ptr(workspace), workspace.numel() *
                                         workspace.element_size(), _stream(stream)))


def oc_suffix_prefill_layer_noalloc(q, k_new, v_new, suffix_tokens: int, pool, layout: Layout, pages,
                                    num_tokens: int, layer: int, out, stream=None) -> None:
    """oc_suffix_prefill_layer without a workspace argument: the library's
    static per-device workspace holds the split partials."""
    bt = make_table(pages, num_tokens)
    kp = make_pool(pool, layout)
    _check(lib().oc_suffix_prefill_layer_noalloc(_ptr(q), _ptr(k_new), _ptr(v_new), suffix_tokens, ctypes.byref(kp),
                                                 ctypes.byref(bt), layer, _ptr(out), _stream(stream)))


# ---------------------------------------------------------------------------
# pipeline
# ---------------------------------------------------------------------------

@dataclass
class Request:
    """One request of a pipeline run (tensors are torch device tensors)."""
    prefix_tokens: int
    suffix_tokens: int
    pages: object                      # device int32 block table (None when prefix_tokens == 0)
    q: object                          # [L][Ts][nq][d] bf16
    k_new: object                      # [L][Ts][nkv][d] bf16
    v_new: object                      # [L][Ts][nkv][d] bf16
    out: object                        # [L][Ts][nq][d] bf16
    chunk_objects: object = None       # host numpy uint16 [N][L * S/2], one chunk object per row
    device_payload: object = None      # device [L][Tp * b] bytes, layer payloads back to back
    layer_compute_s: float = 0.0       # per-layer compute window for the allocation policies
    arrival_s: float = 0.0             # arrival after the run starts (allocation policies only)


def oc_context_create(pool, layout: Layout, mode: int, max_prefix_tokens: int, max_suffix_tokens: int,
                      rate_bytes_per_s: float = 0.0, piece_bytes: int = 0, slots: int = 0,
                      producer_threads: int = 0, timeout_ms: int = 0, fault: int = OC_FAULT_NONE,
                      fault_layer: int = 0, device: int = 0, alloc_policy="fifo", margin_bytes_per_s: float = 0.0,
                      delivery="layerwise", theta_bytes: float = 0.0, emulate_compute: bool = False,
                      append_suffix: bool = False, layer_weights: Optional[LayerWeights] = None,
                      attention_per_request: bool = False, epoch_s: float = 0.0):
    pol = ALLOC_POLICIES[alloc_policy] if isinstance(alloc_policy, str) else int(alloc_policy)
    dv = DELIVERIES[delivery] if isinstance(delivery, str) else int(delivery)
    opts = c_pipeline_opts(mode, rate_bytes_per_s, piece_bytes, slots, producer_threads, timeout_ms, fault,
                           fault_layer, pol, margin_bytes_per_s, dv, theta_bytes, int(bool(emulate_compute)),
                           int(bool(append_suffix)), int(bool(attention_per_request)), None, epoch_s)
    lw = layer_weights.c() if layer_weights is not None else None
    if lw is not None:
        opts.layer_weights = ctypes.cast(ctypes.pointer(lw), c_void_p)     # copied by the library
    kp = make_pool(pool, layout)
    ctx = c_void_p()
    _check(lib().oc_context_create(device, ctypes.byref(kp), ctypes.byref(opts), max_prefix_tokens,
                                   max_suffix_tokens, ctypes.byref(ctx)))
    return ctx


def oc_context_destroy(ctx) -> None:
    lib().oc_context_destroy(ctx)


def oc_pipeline_last_ms(ctx) -> float:
    return lib().oc_pipeline_last_ms(ctx)


def oc_pipeline_run(ctx, requests: Sequence[Request], num_layers: int):
    """Run all layers of all requests; returns one dict of timings per request."""
    n = len(requests)
    creqs = (c_request * n)()
    keep = []
    stats = (c_request_stats * n)()
    arrays = []
    for i, r in enumerate(requests):
        bt = make_table(r.pages, r.prefix_tokens)
        keep.append(bt)
        objs = None
        if r.chunk_objects is not None and r.prefix_tokens > 0:
            co = r.chunk_objects
            if not co.flags["C_CONTIGUOUS"]:
                raise ValueError("chunk_objects must be C-contiguous")
            row = co.strides[0]
            objs = (c_void_p * co.shape[0])(*[co.ctypes.data + j * row for j in range(co.shape[0])])
            keep.append(objs)
        creqs[i] = c_request(r.prefix_tokens, r.suffix_tokens, ctypes.pointer(bt), objs,
                             _ptr(r.device_payload), _ptr(r.q), _ptr(r.k_new), _ptr(r.v_new), _ptr(r.out),
                             r.layer_compute_s, r.arrival_s)
        per = [(c_double * num_layers)() for _ in range(4)]
        arrays.append(per)
        stats[i] = c_request_stats(0.0, *per, 0.0, 0, 0.0)
    _check(lib().oc_pipeline_run(ctx, creqs, n, stats))
    out = []
    for i in range(n):
        p = arrays[i]
        out.append({"ttft_ms": stats[i].ttft_ms, "produced_ms": list(p[0]), "landed_ms": list(p[1]),
                    "ingested_ms": list(p[2]), "done_ms": list(p[3]), "rate_bytes_per_s": stats[i].rate_bytes_per_s,
                    "delivery": {v: k for k, v in DELIVERIES.items()}[stats[i].delivery],
                    "admitted_ms": stats[i].admitted_ms})
    return out


def oc_bandwidth_allocate(policy, layer_bytes, layer_compute_s, budget_bytes_per_s: float,
                          margin_bytes_per_s: float = 0.0):
    """Per-request rates (bytes/s) under a shared budget; `policy` is a name
    of ALLOC_POLICIES or its number."""
    pol = ALLOC_POLICIES.get(policy, -1) if isinstance(policy, str) else int(policy)
    n = len(layer_bytes)
    s = (c_double * n)(*layer_bytes)
    c = (c_double * n)(*layer_compute_s) if layer_compute_s is not None else None
    out = (c_double * n)()
    _check(lib().oc_bandwidth_allocate(pol, n, s, c, budget_bytes_per_s, margin_bytes_per_s, out))
    return list(out)


def oc_epoch_schedule(policy, layer_bytes, layer_compute_s, num_layers: int, arrival_s, budget_bytes_per_s: float,
                      margin_bytes_per_s: float = 0.0, epoch_s: float = 0.0):
    """(rates in bytes/s, admission times in s) of requests arriving at
    arrival_s under scheduling epochs; `policy` as in oc_bandwidth_allocate."""
    pol = ALLOC_POLICIES.get(policy, -1) if isinstance(policy, str) else int(policy)
    n = len(layer_bytes)
    s = (c_double * n)(*layer_bytes)
    c = (c_double * n)(*layer_compute_s) if layer_compute_s is not None else None
    a = (c_double * n)(*arrival_s)
    rates, admit = (c_double * n)(), (c_double * n)()
    _check(lib().oc_epoch_schedule(pol, n, s, c, num_layers, a, budget_bytes_per_s, margin_bytes_per_s, epoch_s,
                                   rates, admit))
    return list(rates), list(admit)
