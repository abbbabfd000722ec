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
