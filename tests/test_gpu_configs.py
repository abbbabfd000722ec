"""GPU parity at the five workloads' full sizes, and at the paper's other
chunk sizes (G = 64, 256), in the kernels' real launch configuration: for
the first and the last layer of every request, the ingest and the suffix
append are compared bit for bit over the whole pool (the full page count,
4x the pages the prefix needs), every whole chunk of prefix and suffix is
offloaded back into chunk objects and compared with the stored ones, and the
attention is checked against the float64 oracle on every suffix row and head
up to a 4K context, and beyond it on 64 sampled suffix rows (always the first
and the last) and every head.  The pool holds two layers, standing in for
layers 0 and L-1."""
import numpy as np
import pytest

import kvgen
import oracle
from tests.gpu_util import SENTINEL, assert_attention_close, from_dev, require_gpu, to_dev

pytestmark = pytest.mark.gpu

N_ROWS = 64           # first and last suffix rows plus seeded ones, per request and layer
FULL_ROWS_CONTEXT = 8192   # up to this prefix + suffix, every suffix row is checked


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


def _suffix_chunk_objects(kn, vn, G, n_suf):
    """Whole suffix chunks as KV_L2TD objects, straight from the dense K/V:
    object s holds, layer by layer, K then V of tokens s*G .. (s+1)*G-1."""
    return np.stack([np.concatenate([np.concatenate([k[s * G:(s + 1) * G].ravel(), v[s * G:(s + 1) * G].ravel()])
                                     for k, v in zip(kn, vn)]) for s in range(n_suf)]) if n_suf else None


def check_workload(wl):
    """Ingest + suffix append of the first and the last layer of every request
    (whole pool bit for bit), offload of every whole chunk of prefix and
    suffix (against the generated objects), then attention on sampled rows."""
    import torch
    import paper_2605_22850_amd as oc
    name = wl.name
    L, nq, nkv, d, G, Ps = (wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.chunk_tokens,
                            wl.page_size)
    layers = [0, L - 1]
    print(f"[config] {name}: L={L} nq={nq} nkv={nkv} d={d} G={G} prefixes={wl.prefix_tokens} "
          f"pool={wl.pool_pages}", flush=True)
    layout = oc.Layout(2, nq, nkv, d, Ps, G, wl.pool_pages)
    # tables hold room for the suffix behind the prefix
    need = [-(-(wl.prefix_tokens[r] + wl.suffix_tokens[r]) // Ps) for r in range(wl.n_requests)]
    tables = kvgen.block_tables(wl.seed, need, wl.pool_pages)
    pool = torch.full((layout.pool_elems,), int(np.uint16(SENTINEL).view(np.int16)), dtype=torch.int16,
                      device="cuda")
    want_pool = np.full(oracle.pool_shape(2, wl.pool_pages, nkv, Ps, d), SENTINEL, dtype=np.uint16)
    slices, suffix = {}, {}
    for r in range(wl.n_requests):
        n, tp, ts = wl.n_chunks(r), wl.prefix_tokens[r], wl.suffix_tokens[r]
        d_table = torch.from_numpy(tables[r]).cuda()
        for li, l in enumerate(layers):
            sl = kvgen.chunk_layer_slices(wl.seed, r, l, n, wl.slice_elems)      # row j = chunk j's slice
            slices[(r, l)] = sl
            oc.oc_kv_layer_ingest(to_dev(sl.reshape(-1)), n, d_table, tp, pool, layout, li)
            oracle.ingest_layer(sl.reshape(-1), n, G, nkv, d, Ps, tables[r], want_pool, li)
            q = kvgen.suffix_tensor(wl.seed, kvgen.KIND_Q, r, l, (ts, nq, d))
            kn = kvgen.suffix_tensor(wl.seed, kvgen.KIND_KNEW, r, l, (ts, nkv, d))
            vn = kvgen.suffix_tensor(wl.seed, kvgen.KIND_VNEW, r, l, (ts, nkv, d))
            suffix[(r, l)] = (q, kn, vn)
            oc.oc_kv_suffix_append(to_dev(kn), to_dev(vn), ts, d_table, tp, pool, layout, li)
            oracle.append_suffix(kn, vn, tp, tables[r], want_pool, li, Ps)
    torch.cuda.synchronize()
    got_pool = from_dev(pool).reshape(want_pool.shape)
    assert np.array_equal(got_pool, want_pool), f"{name}: pool differs from the oracle's scatter + append"
    del got_pool, want_pool

    for r in range(wl.n_requests):
        n, tp, ts = wl.n_chunks(r), wl.prefix_tokens[r], wl.suffix_tokens[r]
        n_suf = ts // G
        total = n + n_suf
        d_table = torch.from_numpy(tables[r]).cuda()
        objs = torch.empty(total * 2 * wl.slice_elems, dtype=torch.int16, device="cuda")
        oc.oc_kv_chunks_gather(d_table, tp + n_suf * G, pool, layout, 0, total, objs)
        torch.cuda.synchronize()
        got = from_dev(objs).reshape(total, 2 * wl.slice_elems)
        assert np.array_equal(got[:n], np.concatenate([slices[(r, l)] for l in layers], axis=1)), \
            f"{name} request {r}: offloaded prefix chunks differ from the stored objects"
        if n_suf:
            want = _suffix_chunk_objects([suffix[(r, l)][1] for l in layers], [suffix[(r, l)][2] for l in layers],
                                         G, n_suf)
            assert np.array_equal(got[n:], want), f"{name} request {r}: offloaded suffix chunks differ"
        print(f"  request {r}: offloaded {n} prefix + {n_suf} suffix chunks", flush=True)
        del objs, got

    for r in range(wl.n_requests):
        tp, ts = wl.prefix_tokens[r], wl.suffix_tokens[r]
        # every row up to a 4K context (tiny, 8b-4k), sampled rows beyond
        rows = list(range(ts)) if tp + ts <= FULL_ROWS_CONTEXT else sample_rows(ts, seed=r)
        d_table = torch.from_numpy(tables[r]).cuda()
        ws = torch.empty(oc.oc_attention_workspace_bytes(layout, tp, ts), dtype=torch.uint8, device="cuda")
        for li, l in enumerate(layers):
            q, kn, vn = suffix[(r, l)]
            out = torch.empty((ts, nq, d), dtype=torch.bfloat16, device="cuda")
            oc.oc_suffix_prefill_layer(to_dev(q, "bf16"), to_dev(kn, "bf16"), to_dev(vn, "bf16"), ts, pool, layout,
                                       d_table, tp, li, out, ws)
            torch.cuda.synchronize()
            sl = slices[(r, l)]
            k, v = oracle.logical_kv([np.ascontiguousarray(sl[j]) for j in range(sl.shape[0])], G, nkv, d, 0)
            ref = oracle.attention(q, k, v, kn, vn, rows=rows)
            err = assert_attention_close(from_dev(out)[rows], ref, f"{name} request {r} layer {l}")
            print(f"  request {r} layer {l}: rows {len(rows)} max|err| {err[0]:.2e} rel L2 {err[1]:.2e}", flush=True)


@pytest.mark.timeout(400)
@pytest.mark.parametrize("name", kvgen.WORKLOADS + kvgen.SHARD_WORKLOADS)
def test_workload_first_and_last_layer(name):
    check_workload(kvgen.workload(name))


@pytest.mark.timeout(400)
@pytest.mark.parametrize("name,G", [("8b-64k", 64), ("8b-64k", 256), ("8b-4k", 64), ("70b-32k", 256)])
def test_paper_chunk_sizes_at_full_size(name, G):
    # the paper's end-to-end settings use G = 64 (main) and 256 besides 16
    check_workload(kvgen.with_chunk_tokens(kvgen.workload(name), G))


@pytest.mark.timeout(600)
def test_batch8_batched_pipeline_launch_at_full_size():
    """The batch workload's own launch configuration: the device-staged
    pipeline with its default attention, one launch per layer over all eight
    requests with the key split planned for all their row tiles together.
    The two pool layers hold the workload's first and last layers; the pool
    is compared bit for bit with the oracle's scatter, and every request's
    attention with the float64 oracle on 64 sampled suffix rows (the first
    and the last among them) and every head."""
    import torch
    import paper_2605_22850_amd as oc
    wl = kvgen.workload("batch8")
    L, nq, nkv, d, G, Ps = (wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.chunk_tokens,
                            wl.page_size)
    layers = [0, L - 1]
    n_req = wl.n_requests
    print(f"[batch8 batched pipeline] prefixes={wl.prefix_tokens} suffix={wl.suffix_tokens} "
          f"pool={wl.pool_pages}", flush=True)
    layout = oc.Layout(2, nq, nkv, d, Ps, G, wl.pool_pages)
    tables = kvgen.block_tables(wl.seed, [wl.pages_needed(r) for r in range(n_req)], wl.pool_pages)
    pool = torch.full((layout.pool_elems,), int(np.uint16(SENTINEL).view(np.int16)), dtype=torch.int16,
                      device="cuda")
    want_pool = np.full(oracle.pool_shape(2, wl.pool_pages, nkv, Ps, d), SENTINEL, dtype=np.uint16)
    reqs, host = [], []
    for r in range(n_req):
        n, tp, ts = wl.n_chunks(r), wl.prefix_tokens[r], wl.suffix_tokens[r]
        sl = [kvgen.chunk_layer_slices(wl.seed, r, l, n, wl.slice_elems) for l in layers]
        for li in range(2):
            oracle.ingest_layer(sl[li].reshape(-1), n, G, nkv, d, Ps, tables[r], want_pool, li)
        sfx = [np.stack([kvgen.suffix_tensor(wl.seed, kind, r, l, shape) for l in layers])
               for kind, shape in ((kvgen.KIND_Q, (ts, nq, d)), (kvgen.KIND_KNEW, (ts, nkv, d)),
                                   (kvgen.KIND_VNEW, (ts, nkv, d)))]
        host.append((sl, sfx))
        payload = to_dev(np.concatenate([s.reshape(-1) for s in sl]))      # layer payloads back to back
        reqs.append(oc.Request(tp, ts, torch.from_numpy(tables[r]).cuda(), to_dev(sfx[0], "bf16"),
                               to_dev(sfx[1], "bf16"), to_dev(sfx[2], "bf16"),
                               torch.zeros((2, ts, nq, d), dtype=torch.bfloat16, device="cuda"),
                               device_payload=payload))
    ctx = oc.oc_context_create(pool, layout, oc.OC_MODE_DEVICE_STAGED, max(wl.prefix_tokens),
                               max(wl.suffix_tokens))
    try:
        stats = oc.oc_pipeline_run(ctx, reqs, 2)
    finally:
        oc.oc_context_destroy(ctx)
    torch.cuda.synchronize()
    for li in range(2):     # one launch per layer: every request's layer is done at the same moment
        assert len({st["done_ms"][li] for st in stats}) == 1, f"layer {li} was not one batched launch"
    assert np.array_equal(from_dev(pool).reshape(want_pool.shape), want_pool), "batch8: pool differs"
    del want_pool
    for r in range(n_req):
        ts = wl.suffix_tokens[r]
        rows = sample_rows(ts, seed=100 + r)
        sl, (q, kn, vn) = host[r]
        got = from_dev(reqs[r].out)
        for li, l in enumerate(layers):
            k, v = oracle.logical_kv([np.ascontiguousarray(s) for s in sl[li]], G, nkv, d, 0)
            ref = oracle.attention(q[li], k, v, kn[li], vn[li], rows=rows)
            err = assert_attention_close(got[li][rows], ref, f"batch8 request {r} layer {l}")
            print(f"  request {r} (T_p {wl.prefix_tokens[r]}) layer {l}: rows {len(rows)} "
                  f"max|err| {err[0]:.2e} rel L2 {err[1]:.2e}", flush=True)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("rate", [0.0, 12.5e9])
def test_producer_pipeline_at_full_size(rate):
    """The 8b-64k request through the host producer at full size: every
    chunk object in host memory, each layer payload assembled from them,
    landed in HBM (in spans of 32 MiB while it is produced, when capped at
    12.5 GB/s; whole, uncapped), ingested (the second layer beside the first
    layer's attention) and attended.  The two pool layers hold the workload's
    first and last layers; the pool is compared bit for bit with the
    oracle's scatter and the attention with the float64 oracle on 64 sampled
    suffix rows and every head.  Capped, the run cannot end before the
    producer's last byte is due at the cap."""
    import torch
    import paper_2605_22850_amd as oc
    wl = kvgen.workload("8b-64k")
    L, nq, nkv, d, G, Ps = (wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.chunk_tokens,
                            wl.page_size)
    layers = [0, L - 1]
    n, tp, ts = wl.n_chunks(0), wl.prefix_tokens[0], wl.suffix_tokens[0]
    print(f"[producer full size] 8b-64k rate {rate / 1e9:g} GB/s: T_p {tp}, T_s {ts}, pool {wl.pool_pages}",
          flush=True)
    layout = oc.Layout(2, nq, nkv, d, Ps, G, wl.pool_pages)
    table = kvgen.block_tables(wl.seed, [wl.pages_needed(0)], wl.pool_pages)[0]
    pool = torch.full((layout.pool_elems,), int(np.uint16(SENTINEL).view(np.int16)), dtype=torch.int16,
                      device="cuda")
    want_pool = np.full(oracle.pool_shape(2, wl.pool_pages, nkv, Ps, d), SENTINEL, dtype=np.uint16)
    sl = [kvgen.chunk_layer_slices(wl.seed, 0, l, n, wl.slice_elems) for l in layers]
    for li in range(2):
        oracle.ingest_layer(sl[li].reshape(-1), n, G, nkv, d, Ps, table, want_pool, li)
    objects = np.ascontiguousarray(np.concatenate(sl, axis=1))          # object j: its two layer slices
    q, kn, vn = [np.stack([kvgen.suffix_tensor(wl.seed, kind, 0, l, shape) for l in layers])
                 for kind, shape in ((kvgen.KIND_Q, (ts, nq, d)), (kvgen.KIND_KNEW, (ts, nkv, d)),
                                     (kvgen.KIND_VNEW, (ts, nkv, d)))]
    req = oc.Request(tp, ts, torch.from_numpy(table).cuda(), to_dev(q, "bf16"), to_dev(kn, "bf16"),
                     to_dev(vn, "bf16"), torch.zeros((2, ts, nq, d), dtype=torch.bfloat16, device="cuda"),
                     chunk_objects=objects)
    ctx = oc.oc_context_create(pool, layout, oc.OC_MODE_PRODUCER, tp, ts, rate_bytes_per_s=rate)
    try:
        stats = oc.oc_pipeline_run(ctx, [req], 2)
    finally:
        oc.oc_context_destroy(ctx)
    torch.cuda.synchronize()
    layer_bytes = tp * 2 * nkv * d * 2
    if rate > 0:
        due_ms = 2 * layer_bytes / rate * 1e3
        print(f"  TTFT {stats[0]['ttft_ms']:.2f} ms, last byte due at {due_ms:.2f} ms", flush=True)
        assert stats[0]["ttft_ms"] >= due_ms, "the producer delivered faster than its cap"
    assert np.array_equal(from_dev(pool).reshape(want_pool.shape), want_pool), "pool differs from the oracle's"
    del want_pool
    rows = sample_rows(ts, seed=7)
    got = from_dev(req.out)
    for li, l in enumerate(layers):
        k, v = oracle.logical_kv([np.ascontiguousarray(s) for s in sl[li]], G, nkv, d, 0)
        ref = oracle.attention(q[li], k, v, kn[li], vn[li], rows=rows)
        err = assert_attention_close(got[li][rows], ref, f"producer 8b-64k layer {l}")
        print(f"  layer {l}: rows {len(rows)} max|err| {err[0]:.2e} rel L2 {err[1]:.2e}", flush=True)
