"""GPU parity at the five workloads' full sizes, in the kernels' real launch
configuration: for the first and the last layer of every request, the ingest
is compared bit for bit over the whole pool (the full page count, 4x the
pages the prefix needs), and the attention on sampled suffix rows (always
the first and the last) against the float64 oracle.  The pool holds two
layers, standing in for layers 0 and L-1."""
import numpy as np
import pytest

import kvgen
import oracle
from tests.gpu_util import SENTINEL, assert_attention_close, from_dev, require_gpu, to_dev

pytestmark = pytest.mark.gpu

N_ROWS = 16


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    import torch
    torch.cuda.synchronize()
    yield
    torch.cuda.synchronize()


def sample_rows(ts, n=N_ROWS, seed=0):
    rng = np.random.default_rng(seed)
    mid = rng.choice(np.arange(1, max(2, ts - 1)), size=min(n - 2, max(0, ts - 2)), replace=False)
    return sorted(set([0, ts - 1, *mid.tolist()]))


@pytest.mark.timeout(400)
@pytest.mark.parametrize("name", kvgen.WORKLOADS)
def test_workload_first_and_last_layer(name):
    import torch
    import paper_2605_22850_amd as oc
    wl = kvgen.workload(name)
    L, nq, nkv, d, G, Ps = (wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.chunk_tokens,
                            wl.page_size)
    layers = [0, L - 1]
    print(f"[config] {name}: L={L} nq={nq} nkv={nkv} d={d} prefixes={wl.prefix_tokens} pool={wl.pool_pages}",
          flush=True)
    layout = oc.Layout(2, nq, nkv, d, Ps, G, wl.pool_pages)
    tables = kvgen.block_tables(wl.seed, [wl.pages_needed(r) for r in range(wl.n_requests)], wl.pool_pages)
    pool = torch.full((layout.pool_elems,), int(np.uint16(SENTINEL).view(np.int16)), dtype=torch.int16,
                      device="cuda")
    want_pool = np.full(oracle.pool_shape(2, wl.pool_pages, nkv, Ps, d), SENTINEL, dtype=np.uint16)
    slices = {}
    for r in range(wl.n_requests):
        n = wl.n_chunks(r)
        d_table = torch.from_numpy(tables[r]).cuda()
        for li, l in enumerate(layers):
            sl = kvgen.chunk_layer_slices(wl.seed, r, l, n, wl.slice_elems)      # row j = chunk j's slice
            slices[(r, l)] = sl
            oc.oc_kv_layer_ingest(to_dev(sl.reshape(-1)), n, d_table, wl.prefix_tokens[r], pool, layout, li)
            oracle.ingest_layer(sl.reshape(-1), n, G, nkv, d, Ps, tables[r], want_pool, li)
    torch.cuda.synchronize()
    got_pool = from_dev(pool).reshape(want_pool.shape)
    assert np.array_equal(got_pool, want_pool), f"{name}: pool differs from the oracle's scatter"
    del got_pool, want_pool

    for r in range(wl.n_requests):
        tp, ts = wl.prefix_tokens[r], wl.suffix_tokens[r]
        rows = sample_rows(ts, seed=r)
        d_table = torch.from_numpy(tables[r]).cuda()
        ws = torch.empty(oc.oc_attention_workspace_bytes(layout, tp, ts), dtype=torch.uint8, device="cuda")
        for li, l in enumerate(layers):
            q = kvgen.suffix_tensor(wl.seed, kvgen.KIND_Q, r, l, (ts, nq, d))
            kn = kvgen.suffix_tensor(wl.seed, kvgen.KIND_KNEW, r, l, (ts, nkv, d))
            vn = kvgen.suffix_tensor(wl.seed, kvgen.KIND_VNEW, r, l, (ts, nkv, d))
            out = torch.empty((ts, nq, d), dtype=torch.bfloat16, device="cuda")
            oc.oc_suffix_prefill_layer(to_dev(q, "bf16"), to_dev(kn, "bf16"), to_dev(vn, "bf16"), ts, pool, layout,
                                       d_table, tp, li, out, ws)
            torch.cuda.synchronize()
            sl = slices[(r, l)]
            k, v = oracle.logical_kv([np.ascontiguousarray(sl[j]) for j in range(sl.shape[0])], G, nkv, d, 0)
            ref = oracle.attention(q, k, v, kn, vn, rows=rows)
            err = assert_attention_close(from_dev(out)[rows], ref, f"{name} request {r} layer {l}")
            print(f"  request {r} layer {l}: rows {len(rows)} max|err| {err[0]:.2e} rel L2 {err[1]:.2e}", flush=True)
