"""GPU parity of the write path against the oracle: the suffix append (the
full KV state behind the prefix) and the offload gather of whole chunk
objects, as single calls and inside the pipeline.  Pools start filled with a
NaN sentinel and are compared bit for bit; offloaded objects are compared
with the stored ones and with the oracle's gather."""
import zlib

import numpy as np
import pytest

import kvgen
import oracle
from tests.gpu_util import SENTINEL, RequestSet, assert_attention_close, from_dev, require_gpu, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    import torch
    torch.cuda.synchronize()
    yield
    torch.cuda.synchronize()


# (nq, nkv, d, G, Ps, Tp, Ts, P, L)
CASES = {
    "tiny": (4, 2, 64, 16, 16, 256, 32, 64, 2),
    "suffix-starts-mid-page": (8, 2, 128, 8, 16, 40, 29, 32, 3),
    "no-prefix": (4, 4, 64, 16, 16, 0, 19, 8, 1),
    "g64-ragged-tail": (8, 8, 128, 64, 16, 192, 77, 64, 2),
    "g256": (8, 8, 128, 256, 16, 512, 300, 128, 2),
    "odd-heads-d64": (6, 3, 64, 32, 16, 96, 45, 40, 2),
}


@pytest.mark.parametrize("name", list(CASES))
def test_append_and_offload_match_oracle(name):
    import torch
    import paper_2605_22850_amd as oc
    nq, nkv, d, G, Ps, Tp, Ts, P, L = CASES[name]
    seed = zlib.crc32(name.encode()) & 0xFFFF
    print(f"[writeback] {name}", flush=True)
    layout = oc.Layout(L, nq, nkv, d, Ps, G, P)
    slice_elems = 2 * G * nkv * d
    N = Tp // G
    objs = kvgen.chunk_objects(seed, 0, L, N, slice_elems)                  # [N][L][slice]
    table = kvgen.block_tables(seed, [-(-(Tp + Ts) // Ps)], P)[0]
    d_table = torch.from_numpy(table.copy()).cuda()
    k = [kvgen.suffix_tensor(seed, kvgen.KIND_KNEW, 0, l, (Ts, nkv, d)) for l in range(L)]
    v = [kvgen.suffix_tensor(seed, kvgen.KIND_VNEW, 0, l, (Ts, nkv, d)) for l in range(L)]
    pool = torch.full((layout.pool_elems,), int(np.uint16(SENTINEL).view(np.int16)), dtype=torch.int16,
                      device="cuda")
    if N:
        oc.oc_kv_chunks_ingest(to_dev(objs.reshape(-1)), N, 0, d_table, Tp, pool, layout)
    for l in range(L):
        oc.oc_kv_suffix_append(to_dev(k[l]), to_dev(v[l]), Ts, d_table, Tp, pool, layout, l)
    torch.cuda.synchronize()

    want = np.full(oracle.pool_shape(L, P, nkv, Ps, d), SENTINEL, dtype=np.uint16)
    chunks = [np.ascontiguousarray(objs[j]).view(np.uint8).reshape(-1) for j in range(N)]
    for l in range(L):
        if N:
            oracle.ingest_layer(oracle.assemble_layer(chunks, slice_elems * 2, l), N, G, nkv, d, Ps, table, want, l)
        oracle.append_suffix(k[l], v[l], Tp, table, want, l, Ps)
    got = from_dev(pool).reshape(want.shape)
    assert np.array_equal(got, want), "pool differs from the oracle's scatter + append"

    # offload every whole chunk of prefix and suffix
    n_all = (Tp + Ts) // G
    out = torch.full((max(1, n_all) * L * slice_elems,), -1, dtype=torch.int16, device="cuda")
    oc.oc_kv_chunks_gather(d_table, n_all * G, pool, layout, 0, n_all, out)
    torch.cuda.synchronize()
    got_objs = from_dev(out)[:n_all * L * slice_elems].reshape(n_all, L * slice_elems)
    assert np.array_equal(got_objs, oracle.gather_chunks(want, table, 0, n_all, G, nkv, d, Ps))
    assert np.array_equal(got_objs[:N], objs.reshape(N, L * slice_elems)), \
        "offloaded prefix chunks differ from the stored ones"
    # a window of chunks from the middle lands at the start of the output
    if n_all >= 3:
        out.fill_(-1)
        oc.oc_kv_chunks_gather(d_table, n_all * G, pool, layout, 1, n_all - 2, out)
        torch.cuda.synchronize()
        mid = from_dev(out)[:(n_all - 2) * L * slice_elems].reshape(n_all - 2, -1)
        assert np.array_equal(mid, got_objs[1:n_all - 1])
        assert (from_dev(out)[(n_all - 2) * L * slice_elems:] == 0xFFFF).all(), "wrote past the chunks asked for"

    # the per-layer gather reads the prefix back into the layer payload
    for l in range(L):
        if not N:
            break
        lay = torch.empty(N * slice_elems, dtype=torch.int16, device="cuda")
        oc.oc_kv_layer_gather(d_table, Tp, pool, layout, l, lay, N)
        torch.cuda.synchronize()
        assert np.array_equal(from_dev(lay), np.ascontiguousarray(objs[:, l, :]).reshape(-1)), f"layer {l}"


def _run(rs, mode, **kw):
    import paper_2605_22850_amd as oc
    ctx = rs.context(mode, **kw)
    try:
        return oc.oc_pipeline_run(ctx, rs.reqs, rs.L)
    finally:
        oc.oc_context_destroy(ctx)


def test_pipeline_appends_every_layer_and_keeps_outputs():
    import paper_2605_22850_amd as oc
    print("[writeback] pipeline append, three requests", flush=True)
    rs = RequestSet(3, 8, 2, 128, [96, 0, 208], [21, 33, 64], 128, seed=9, suffix_room=True).upload(
        with_payload=True)
    # one attention launch per request throughout, so every run (chunkwise
    # requests always get their own) compares bit for bit
    _run(rs, oc.OC_MODE_DEVICE_STAGED, attention_per_request=True)
    base = [from_dev(r.out) for r in rs.reqs]
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())
    want = rs.expected_pool(appended=True)
    for name, mode, kw in (("staged", oc.OC_MODE_DEVICE_STAGED, {}),
                           ("producer", oc.OC_MODE_PRODUCER, {}),
                           ("chunkwise", oc.OC_MODE_PRODUCER, {"delivery": "chunkwise"})):
        rs.d_pool.fill_(np.int16(np.uint16(SENTINEL).view(np.int16)))
        for r in rs.reqs:
            r.out.zero_()
        _run(rs, mode, append_suffix=True, attention_per_request=True, **kw)
        assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), want), name
        for r, req in enumerate(rs.reqs):
            assert np.array_equal(from_dev(req.out), base[r]), f"{name}: request {r} output changed"
    for r in range(3):
        assert_attention_close(base[r][rs.L - 1], rs.expected_out(r, rs.L - 1), f"request {r}")


def test_pipeline_append_needs_room_in_the_table():
    import paper_2605_22850_amd as oc
    print("[writeback] pipeline append validation", flush=True)
    rs = RequestSet(2, 4, 2, 64, [256], [32], 64, seed=4).upload(with_payload=True)
    with pytest.raises(oc.OcError) as e:
        _run(rs, oc.OC_MODE_DEVICE_STAGED, append_suffix=True)
    assert e.value.status == oc._lib.OC_ERANGE
    assert "suffix" in str(e.value)
