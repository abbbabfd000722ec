"""Test-side helpers: build seeded single-layer cases, move them to the GPU,
and compute the oracle's expectations.  Inputs come only from kvgen;
expectations only from the oracle."""
from __future__ import annotations

import numpy as np

import kvgen
import oracle

SENTINEL = 0x7FC5            # a NaN bit pattern: must survive where nothing is written
ATOL, RTOL_L2 = 2e-2, 5e-3   # attention tolerance: max |err| and ||err||_2 / ||ref||_2


def require_gpu():
    import pytest
    import torch
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")


def to_dev(a_u16: np.ndarray, dtype=None):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a_u16).view(np.int16).copy()).cuda()
    return t.view(torch.bfloat16) if dtype == "bf16" else t


def from_dev(t) -> np.ndarray:
    import torch
    if t.dtype == torch.bfloat16:
        t = t.view(torch.int16)
    return t.cpu().numpy().view(np.uint16)


class LayerCase:
    """One layer of one request: chunk-object slices, a block table, suffix tensors."""

    def __init__(self, nq, nkv, d, G, Ps, n_chunks, Ts, P, L=2, layer=1, seed=1, table=None, req=0):
        from paper_2605_22850_amd import Layout
        self.nq, self.nkv, self.d, self.G, self.Ps = nq, nkv, d, G, Ps
        self.n_chunks, self.Ts, self.P, self.L, self.layer, self.seed = n_chunks, Ts, P, L, layer, seed
        self.Tp = n_chunks * G
        self.layout = Layout(L, nq, nkv, d, Ps, G, P)
        self.slices = kvgen.chunk_layer_slices(seed, req, layer, n_chunks, 2 * G * nkv * d)
        # the layer payload: every chunk's layer slice, in prefix order
        self.staging = self.slices.reshape(-1)
        need = -(-self.Tp // Ps)
        self.table = (np.asarray(table, dtype=np.int32) if table is not None
                      else kvgen.block_tables(seed, [need], P)[0])
        self.q = kvgen.suffix_tensor(seed, kvgen.KIND_Q, req, layer, (Ts, nq, d))
        self.k_new = kvgen.suffix_tensor(seed, kvgen.KIND_KNEW, req, layer, (Ts, nkv, d))
        self.v_new = kvgen.suffix_tensor(seed, kvgen.KIND_VNEW, req, layer, (Ts, nkv, d))

    def pool_shape(self):
        return oracle.pool_shape(self.L, self.P, self.nkv, self.Ps, self.d)

    def expected_pool(self, fill=SENTINEL):
        pool = np.full(self.pool_shape(), fill, dtype=np.uint16)
        if self.n_chunks:
            oracle.ingest_layer(self.staging, self.n_chunks, self.G, self.nkv, self.d, self.Ps, self.table, pool,
                                self.layer)
        return pool

    def logical_kv(self):
        if self.n_chunks == 0:
            z = np.zeros((0, self.nkv, self.d), np.uint16)
            return z, z
        objs = [np.ascontiguousarray(self.slices[j]) for j in range(self.n_chunks)]
        return oracle.logical_kv(objs, self.G, self.nkv, self.d, 0)

    def expected_attention(self, rows=None):
        k, v = self.logical_kv()
        return oracle.attention(self.q, k, v, self.k_new, self.v_new, rows=rows)

    # ---- GPU side ----
    def upload(self, fill=SENTINEL):
        import torch
        self.d_pool = torch.full((int(np.prod(self.pool_shape())),), np.int16(np.uint16(fill).view(np.int16)),
                                 dtype=torch.int16, device="cuda")
        self.d_staging = to_dev(self.staging) if self.n_chunks else torch.empty(8, dtype=torch.int16, device="cuda")
        self.d_table = torch.from_numpy(self.table.copy()).cuda() if self.table.size else None
        self.d_q = to_dev(self.q, "bf16")
        self.d_k = to_dev(self.k_new, "bf16")
        self.d_v = to_dev(self.v_new, "bf16")
        return self

    def run_ingest(self, stream=None):
        from paper_2605_22850_amd import oc_kv_layer_ingest
        oc_kv_layer_ingest(self.d_staging, self.n_chunks, self.d_table, self.Tp, self.d_pool, self.layout,
                           self.layer, stream)

    def run_attention(self, stream=None, table=None):
        import torch
        from paper_2605_22850_amd import oc_attention_workspace_bytes, oc_suffix_prefill_layer
        nbytes = oc_attention_workspace_bytes(self.layout, self.Tp, self.Ts)
        ws = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
        out = torch.empty((self.Ts, self.nq, self.d), dtype=torch.bfloat16, device="cuda")
        oc_suffix_prefill_layer(self.d_q, self.d_k, self.d_v, self.Ts, self.d_pool, self.layout,
                                self.d_table if table is None else table, self.Tp, self.layer, out, ws, stream)
        return out


def attention_errors(got_bf16: np.ndarray, ref: np.ndarray):
    g = (got_bf16.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    err = g - ref
    max_abs = float(np.abs(err).max()) if err.size else 0.0
    rel = float(np.linalg.norm(err) / max(np.linalg.norm(ref), 1e-300))
    return max_abs, rel


def assert_attention_close(got_bf16: np.ndarray, ref: np.ndarray, what=""):
    max_abs, rel = attention_errors(got_bf16, ref)
    assert np.isfinite(max_abs) and max_abs <= ATOL and rel <= RTOL_L2, \
        f"{what}: max|err|={max_abs:.3e} (<= {ATOL}), rel L2={rel:.3e} (<= {RTOL_L2})"
    return max_abs, rel


class RequestSet:
    """Several requests sharing one pool, every layer: chunk objects, block
    tables and per-layer suffix tensors, all from kvgen."""

    def __init__(self, L, nq, nkv, d, prefix_tokens, suffix_tokens, pool_pages, seed=1, G=16, Ps=16,
                 suffix_room=False):
        from paper_2605_22850_amd import Layout
        self.L, self.nq, self.nkv, self.d, self.G, self.Ps = L, nq, nkv, d, G, Ps
        self.prefix, self.suffix, self.P, self.seed = list(prefix_tokens), list(suffix_tokens), pool_pages, seed
        self.layout = Layout(L, nq, nkv, d, Ps, G, pool_pages)
        self.slice_elems = 2 * G * nkv * d
        self.objs = [kvgen.chunk_objects(seed, r, L, tp // G, self.slice_elems) for r, tp in enumerate(self.prefix)]
        # with suffix_room the tables also hold the pages the suffix is appended to
        self.suffix_room = suffix_room
        self.tables = kvgen.block_tables(seed, [-(-(tp + (ts if suffix_room else 0)) // Ps)
                                                for tp, ts in zip(self.prefix, self.suffix)], pool_pages)
        self.q, self.k_new, self.v_new = [], [], []
        for r, ts in enumerate(self.suffix):
            self.q.append(np.stack([kvgen.suffix_tensor(seed, kvgen.KIND_Q, r, l, (ts, nq, d)) for l in range(L)]))
            self.k_new.append(np.stack([kvgen.suffix_tensor(seed, kvgen.KIND_KNEW, r, l, (ts, nkv, d))
                                        for l in range(L)]))
            self.v_new.append(np.stack([kvgen.suffix_tensor(seed, kvgen.KIND_VNEW, r, l, (ts, nkv, d))
                                        for l in range(L)]))

    def chunk_rows(self, r):
        # one row per chunk object: the object's L slices back to back
        return self.objs[r].reshape(self.objs[r].shape[0], self.L * self.slice_elems)

    def pool_shape(self):
        return oracle.pool_shape(self.L, self.P, self.nkv, self.Ps, self.d)

    def expected_pool(self, fill=SENTINEL, layers=None, appended=False):
        pool = np.full(self.pool_shape(), fill, dtype=np.uint16)
        for r, tp in enumerate(self.prefix):
            if appended:
                for l in (range(self.L) if layers is None else layers):
                    oracle.append_suffix(self.k_new[r][l], self.v_new[r][l], tp, self.tables[r], pool, l, self.Ps)
            if tp == 0:
                continue
            chunks = [np.ascontiguousarray(self.objs[r][j]).view(np.uint8).reshape(-1)
                      for j in range(self.objs[r].shape[0])]
            for l in (range(self.L) if layers is None else layers):
                staging = oracle.assemble_layer(chunks, self.slice_elems * 2, l)
                oracle.ingest_layer(staging, tp // self.G, self.G, self.nkv, self.d, self.Ps, self.tables[r], pool, l)
        return pool

    def expected_out(self, r, l, rows=None):
        chunks = [np.ascontiguousarray(self.objs[r][j]).reshape(-1) for j in range(self.objs[r].shape[0])]
        if chunks:
            k, v = oracle.logical_kv(chunks, self.G, self.nkv, self.d, l)
        else:
            k = v = np.zeros((0, self.nkv, self.d), np.uint16)
        return oracle.attention(self.q[r][l], k, v, self.k_new[r][l], self.v_new[r][l], rows=rows)

    def upload(self, fill=SENTINEL, with_payload=False):
        import torch
        from paper_2605_22850_amd import Request
        self.d_pool = torch.full((int(np.prod(self.pool_shape())),), np.int16(np.uint16(fill).view(np.int16)),
                                 dtype=torch.int16, device="cuda")
        self.reqs = []
        for r, (tp, ts) in enumerate(zip(self.prefix, self.suffix)):
            pages = torch.from_numpy(self.tables[r].copy()).cuda() if self.tables[r].size else None
            payload = None
            if with_payload and tp:
                # layer-major payloads: layer l = every chunk's slice l, in prefix order
                payload = to_dev(np.ascontiguousarray(self.objs[r].transpose(1, 0, 2)).reshape(-1))
            out = torch.zeros((self.L, ts, self.nq, self.d), dtype=torch.bfloat16, device="cuda")
            self.reqs.append(Request(tp, ts, pages, to_dev(self.q[r], "bf16"), to_dev(self.k_new[r], "bf16"),
                                     to_dev(self.v_new[r], "bf16"), out, chunk_objects=self.chunk_rows(r),
                                     device_payload=payload))
        return self

    def context(self, mode, **kw):
        from paper_2605_22850_amd import oc_context_create
        return oc_context_create(self.d_pool, self.layout, mode, max(self.prefix), max(self.suffix), **kw)
