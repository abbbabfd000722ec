"""GPU tests of chunkwise delivery (eq. (2) below the threshold): whole chunk
objects scattered into every layer of the pool match the oracle bit for bit;
a pipeline run that delivers chunkwise (one or several object groups per
request) gives the same pool and the same attention outputs as the
layerwise run, and computes only after the last object is in; the eq. (2)
switch picks each request's delivery by its payload size."""
import numpy as np
import pytest

from tests.gpu_util import SENTINEL, RequestSet, assert_attention_close, from_dev, require_gpu, to_dev

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    import torch
    torch.cuda.synchronize()
    yield
    torch.cuda.synchronize()


def _pool_of(rs):
    return from_dev(rs.d_pool).reshape(rs.pool_shape())


def _fill(rs):
    rs.d_pool.fill_(np.int16(np.uint16(SENTINEL).view(np.int16)))


def _run(rs, mode, **kw):
    import paper_2605_22850_amd as oc
    ctx = rs.context(mode, **kw)
    try:
        return oc.oc_pipeline_run(ctx, rs.reqs, rs.L)
    finally:
        oc.oc_context_destroy(ctx)


@pytest.mark.parametrize("shape", [
    # (L, n_kv, d, G, page, prefix tokens, groups)
    (2, 2, 64, 16, 16, 256, [16]),                 # tiny, one call
    (3, 2, 64, 16, 16, 256, [5, 7, 4]),            # ragged groups: first_chunk offsets
    (2, 4, 128, 64, 16, 320, [2, 3]),              # one chunk spans four pages
    (2, 2, 64, 8, 16, 200, [10, 15]),              # two chunks share a page, partial last page
    (2, 2, 64, 24, 16, 264, [11]),                 # non-power-of-two chunk size
], ids=["tiny", "ragged-groups", "chunk-spans-pages", "chunks-share-page", "g24"])
def test_chunks_ingest_matches_oracle(shape):
    import paper_2605_22850_amd as oc
    L, nkv, d, G, Ps, tp, groups = shape
    print(f"[chunkwise] ingest {shape}", flush=True)
    rs = RequestSet(L, nkv, nkv, d, [tp], [1], 4 * (-(-tp // Ps)), seed=11, G=G, Ps=Ps).upload()
    want = rs.expected_pool()
    objs = np.ascontiguousarray(rs.objs[0])                 # [N][L][S/2] as stored
    j0 = 0
    for n in groups:
        dev = to_dev(objs[j0:j0 + n].reshape(-1))
        oc.oc_kv_chunks_ingest(dev, n, j0, rs.reqs[0].pages, tp, rs.d_pool, rs.layout)
        j0 += n
    assert j0 == tp // G
    assert np.array_equal(_pool_of(rs), want)


def test_pipeline_chunkwise_matches_layerwise():
    import paper_2605_22850_amd as oc
    print("[chunkwise] pipeline tiny: two object groups", flush=True)
    rs = RequestSet(2, 4, 2, 64, [256], [32], 64, seed=1).upload()
    want = rs.expected_pool()
    _fill(rs)
    lw = _run(rs, oc.OC_MODE_PRODUCER)
    lw_out = from_dev(rs.reqs[0].out)
    assert np.array_equal(_pool_of(rs), want)
    _fill(rs)
    rs.reqs[0].out.zero_()
    cw = _run(rs, oc.OC_MODE_PRODUCER, delivery="chunkwise", rate_bytes_per_s=20e6, piece_bytes=4096)
    assert np.array_equal(_pool_of(rs), want)
    cw_out = from_dev(rs.reqs[0].out)
    assert np.array_equal(cw_out, lw_out)
    for l in range(rs.L):
        assert_attention_close(cw_out[l], rs.expected_out(0, l), f"layer {l}")
    st = cw[0]
    assert st["delivery"] == "chunkwise" and lw[0]["delivery"] == "layerwise"
    # every layer became usable with the last object group and computes after it
    last_in = max(st["ingested_ms"])
    assert all(abs(t - last_in) < 1e-9 for t in st["ingested_ms"])
    assert min(st["done_ms"]) >= last_in
    # paced: the whole payload (every object) takes bytes / rate to arrive
    total = rs.L * 256 * 2 * 2 * 64 * 2
    assert max(st["produced_ms"]) >= 0.95 * total / 20e6 * 1e3


def test_pipeline_chunkwise_many_groups_and_requests():
    # two requests sharing a pool, each split over several object groups
    # (a slot holds N_max/L objects), plus a third with no cached prefix
    import paper_2605_22850_amd as oc
    print("[chunkwise] pipeline 3 requests, 4 layers", flush=True)
    rs = RequestSet(4, 8, 2, 128, [384, 160, 0], [24, 9, 5], 4 * 40, seed=5).upload()
    want = rs.expected_pool()
    _fill(rs)
    stats = _run(rs, oc.OC_MODE_PRODUCER, delivery="chunkwise", slots=2, producer_threads=3)
    assert np.array_equal(_pool_of(rs), want)
    for r in range(3):
        out = from_dev(rs.reqs[r].out)
        for l in range(rs.L):
            assert_attention_close(out[l], rs.expected_out(r, l), f"request {r} layer {l}")
    assert [s["delivery"] for s in stats] == ["chunkwise", "chunkwise", "layerwise"]


def test_eq2_switch_per_request():
    # theta between the two payloads: the small request goes chunkwise, the
    # large one layerwise; results do not depend on the delivery
    import paper_2605_22850_amd as oc
    print("[chunkwise] eq. (2) switch", flush=True)
    rs = RequestSet(2, 4, 2, 64, [128, 512], [16, 16], 4 * 48, seed=9).upload()
    b_obj = rs.L * 2 * 16 * 2 * 64 * 2                     # L * S
    W = [tp // 16 * b_obj for tp in rs.prefix]
    theta = (W[0] + W[1]) / 2
    want = rs.expected_pool()
    _fill(rs)
    stats = _run(rs, oc.OC_MODE_PRODUCER, delivery="auto", theta_bytes=theta, rate_bytes_per_s=40e6)
    assert [s["delivery"] for s in stats] == ["chunkwise", "layerwise"]
    assert np.array_equal(_pool_of(rs), want)
    for r in range(2):
        out = from_dev(rs.reqs[r].out)
        for l in range(rs.L):
            assert_attention_close(out[l], rs.expected_out(r, l), f"request {r} layer {l}")
    # at theta 0 everything is layerwise, above both payloads everything chunkwise
    stats = _run(rs, oc.OC_MODE_PRODUCER, delivery="auto", theta_bytes=0.0)
    assert [s["delivery"] for s in stats] == ["layerwise", "layerwise"]
    stats = _run(rs, oc.OC_MODE_PRODUCER, delivery="auto", theta_bytes=2.0 * W[1])
    assert [s["delivery"] for s in stats] == ["chunkwise", "chunkwise"]


def test_chunkwise_delivery_validation():
    import paper_2605_22850_amd as oc
    rs = RequestSet(2, 4, 2, 64, [256], [32], 64, seed=1).upload()
    with pytest.raises(oc.OcError) as e:
        rs.context(oc.OC_MODE_PRODUCER, delivery="chunkwise", alloc_policy="equal", rate_bytes_per_s=1e9)
    assert e.value.status == oc._lib.OC_EINVAL
    with pytest.raises(oc.OcError):
        rs.context(oc.OC_MODE_PRODUCER, delivery=7)
    with pytest.raises(oc.OcError):
        rs.context(oc.OC_MODE_PRODUCER, delivery="auto", theta_bytes=-1.0)
    # auto + a policy is fine while every request lands on the layerwise side,
    # and an error once one falls below theta
    rs.reqs[0].layer_compute_s = 0.01
    ctx = rs.context(oc.OC_MODE_PRODUCER, delivery="auto", theta_bytes=1e12, alloc_policy="equal",
                     rate_bytes_per_s=1e9)
    try:
        with pytest.raises(oc.OcError) as e:
            oc.oc_pipeline_run(ctx, rs.reqs, rs.L)
        assert b"chunkwise" in str(e.value).encode()
    finally:
        oc.oc_context_destroy(ctx)


# (G, Ps, n_chunks, nkv, d, L): whole chunk objects into pools whose pages are
# not 16 slots, or whose head rows the attention does not take
OBJECT_SHAPE_CASES = [(8, 24, 17, 2, 64, 3), (40, 8, 5, 3, 96, 2), (16, 32, 9, 8, 128, 4), (24, 48, 6, 1, 256, 2)]


@pytest.mark.parametrize("G,Ps,n,nkv,d,L", OBJECT_SHAPE_CASES)
def test_chunk_objects_at_other_page_and_head_sizes(G, Ps, n, nkv, d, L):
    """Every layer of whole chunk objects in one call, first all of them and
    then a range starting mid-prefix on a fresh pool: the pool equals the
    oracle's per-layer scatter bit for bit, and the offload gather of the
    same range returns the stored objects."""
    import torch
    import kvgen
    import oracle
    import paper_2605_22850_amd as oc
    print(f"[chunk objects] G {G} Ps {Ps} chunks {n} nkv {nkv} d {d} L {L}", flush=True)
    Tp = n * G
    need = -(-Tp // Ps)
    P = need + 3
    slice_elems = 2 * G * nkv * d
    objs = kvgen.chunk_objects(Ps * 31 + G, 0, L, n, slice_elems)          # [n][L][S/2]
    table = kvgen.block_tables(Ps * 31 + G, [need], P)[0]
    layout = oc.Layout(L, 2 * nkv, nkv, d, Ps, G, P)
    d_table = torch.from_numpy(table.copy()).cuda()
    for first, count in ((0, n), (n // 3, n - n // 3 - 1)):
        pool = torch.full((layout.pool_elems,), int(np.uint16(SENTINEL).view(np.int16)), dtype=torch.int16,
                          device="cuda")
        want = np.full(oracle.pool_shape(L, P, nkv, Ps, d), SENTINEL, dtype=np.uint16)
        part = np.ascontiguousarray(objs[first:first + count])
        for l in range(L):
            # the oracle scatters the range as the layer payload of chunks first .. first+count-1:
            # its tokens start at first * G, so it runs over a table shifted by those tokens' pages
            full = np.full((n, slice_elems), 0, dtype=np.uint16)
            full[first:first + count] = part[:, l, :]
            ref = np.full(oracle.pool_shape(L, P, nkv, Ps, d), SENTINEL, dtype=np.uint16)
            oracle.ingest_layer(full.reshape(-1), n, G, nkv, d, Ps, table, ref, l)
            # keep only the slots of tokens first*G .. (first+count)*G - 1
            for T in range(first * G, (first + count) * G):
                page, slot = table[T // Ps], T % Ps
                want[l, :, page, :, slot * d:(slot + 1) * d] = ref[l, :, page, :, slot * d:(slot + 1) * d]
        oc.oc_kv_chunks_ingest(to_dev(part.reshape(-1)), count, first, d_table, Tp, pool, layout)
        out = torch.empty(count * L * slice_elems, dtype=torch.int16, device="cuda")
        oc.oc_kv_chunks_gather(d_table, Tp, pool, layout, first, count, out)
        torch.cuda.synchronize()
        assert np.array_equal(from_dev(pool).reshape(want.shape), want), f"pool differs (chunks {first}+{count})"
        assert np.array_equal(from_dev(out).reshape(part.shape), part), f"gather differs (chunks {first}+{count})"
