"""Pins for the CPU oracle: it is checked against what the paper and the
mathematics fix, never against itself or the GPU path."""
import math

import numpy as np
import pytest
import torch

import kvgen
import oracle
from tests.conftest import golden_rows


def rand_bf16(rng, shape, scale=1.0):
    return kvgen.f32_to_bf16_bits((rng.standard_normal(shape) * scale).astype(np.float32))


def f64(b):
    return kvgen.bf16_bits_to_f32(b).astype(np.float64)


# ---------------------------------------------------------------------------
# layer assembly (Section 3.3, layerwise GET)
# ---------------------------------------------------------------------------

def test_assemble_matches_hand_worked_layerwise_get():
    rows = golden_rows("layerwise_get_tiny.txt")
    objs = [np.array([int(x) for x in r[2:]], dtype=np.uint8) for r in rows if r[0] == "object"]
    want = {int(r[1].rstrip(":")): [int(x) for x in r[2:]] for r in rows if r[0] == "layer"}
    for layer, expect in want.items():
        got = oracle.assemble_layer(objs, 2, layer)
        assert got.tolist() == expect


def test_assemble_only_reads_the_layer_range():
    # every byte of B_l must come from [l*S, (l+1)*S) of its own object, in object order
    n, L, S = 5, 3, 8
    objs = [np.arange(L * S, dtype=np.uint8) + np.uint8(50 * j) for j in range(n)]
    for layer in range(L):
        got = oracle.assemble_layer(objs, S, layer).reshape(n, S)
        for j in range(n):
            src = (got[j].astype(int) - 50 * j)
            assert src.min() >= layer * S and src.max() < (layer + 1) * S
            assert (np.diff(src) == 1).all()


# ---------------------------------------------------------------------------
# KV_L2TD decoding (Section 3.3)
# ---------------------------------------------------------------------------

def test_kv_l2td_positions_match_hand_worked_object():
    L, G, nkv, d = 2, 2, 2, 2
    obj = np.arange(L * 2 * G * nkv * d, dtype=np.uint16)
    for r in golden_rows("kv_l2td_positions.txt"):
        layer, mat, t, h, e, idx = int(r[0]), r[1], int(r[2]), int(r[3]), int(r[4]), int(r[5])
        k, v = oracle.logical_kv([obj], G, nkv, d, layer)
        got = (k if mat == "K" else v)[t, h, e]
        assert int(got) == idx, (r, int(got))


def test_layer_slice_is_eq1_bytes_and_self_contained():
    # eq. (1): S = 2 G n_kv d p; decoding layer l touches only that slice
    L, G, nkv, d = 3, 4, 2, 8
    S_elems = 2 * G * nkv * d
    obj = np.arange(L * S_elems, dtype=np.uint16)
    for layer in range(L):
        k, v = oracle.logical_kv([obj], G, nkv, d, layer)
        vals = np.concatenate([k.ravel(), v.ravel()])
        assert vals.min() == layer * S_elems and vals.max() == (layer + 1) * S_elems - 1
        assert np.unique(vals).size == S_elems          # a bijection onto the slice
        assert k.max() < v.min()                         # K matrix precedes V


# ---------------------------------------------------------------------------
# scatter / gather through the block table
# ---------------------------------------------------------------------------

SENTINEL = 0xBEEF


def _numpy_scatter(staging, n_chunks, G, nkv, d, Ps, table, pool, layer):
    """Independent formulation: reshape + fancy indexing.  The block table
    maps logical token T to (page table[T // Ps], slot T % Ps); K and V
    pages are [slot][dim]."""
    L, _, P = pool.shape[:3]
    x = staging.reshape(n_chunks, 2, G, nkv, d).transpose(1, 0, 2, 3, 4).reshape(2, n_chunks * G, nkv, d)
    T = np.arange(n_chunks * G)
    pages, slots = table[T // Ps], T % Ps
    view = pool.reshape(L, 2, P, nkv, Ps, d)
    view[layer, 0, pages, :, slots, :] = x[0]
    view[layer, 1, pages, :, slots, :] = x[1]


@pytest.mark.parametrize("G,Ps,n_chunks,nkv,d", [
    (16, 16, 5, 2, 64),      # one chunk per page
    (8, 16, 5, 2, 8),        # two chunks per page, last page half full
    (32, 16, 3, 1, 16),      # two pages per chunk
    (16, 16, 1, 8, 128),     # Llama-shaped page
    (8, 8, 7, 2, 16),        # page of 8 slots
    (16, 24, 5, 2, 8),       # page size not a power of two, chunks straddle pages
    (40, 24, 3, 1, 16),      # chunks longer than a page, neither divides the other
    (8, 32, 9, 4, 8),        # four chunks per page, last page partial
])
def test_ingest_matches_numpy_formulation(G, Ps, n_chunks, nkv, d):
    rng = np.random.default_rng(7)
    L, P, layer = 3, 16, 1
    staging = rng.integers(0, 1 << 16, n_chunks * 2 * G * nkv * d, dtype=np.uint16)
    pages_needed = -(-n_chunks * G // Ps)
    table = rng.permutation(P)[:pages_needed].astype(np.int32)
    pool = np.full(oracle.pool_shape(L, P, nkv, Ps, d), SENTINEL, dtype=np.uint16)
    ref = pool.copy()
    oracle.ingest_layer(staging, n_chunks, G, nkv, d, Ps, table, pool, layer)
    _numpy_scatter(staging, n_chunks, G, nkv, d, Ps, table, ref, layer)
    assert np.array_equal(pool, ref)
    # untouched: other layers, pages outside the table, slots past the prefix
    assert (pool[[0, 2]] == SENTINEL).all()
    other = np.setdiff1d(np.arange(P), table)
    assert (pool[layer][:, other] == SENTINEL).all()
    written = (pool != SENTINEL).sum()
    assert written <= staging.size
    # gather undoes scatter
    back = oracle.gather_layer(pool, layer, table, n_chunks, G, nkv, d, Ps)
    assert np.array_equal(back, staging)
    # the threaded form (the CPU baseline's) gives the same pool, for thread
    # counts that split the chunks evenly, unevenly and beyond their number
    for threads in (2, 3, 8):
        mt = np.full(oracle.pool_shape(L, P, nkv, Ps, d), SENTINEL, dtype=np.uint16)
        oracle.ingest_layer(staging, n_chunks, G, nkv, d, Ps, table, mt, layer, threads=threads)
        assert np.array_equal(mt, ref), threads


def test_paged_read_returns_logical_token():
    # what paging means: the K (V) of logical token T, head h, dim e is found in
    # page table[T // Ps] at slot T % Ps -- checked from the decoded chunk objects
    G = Ps = 16
    L, nkv, d, n_chunks, P = 2, 2, 8, 4, 10
    rng = np.random.default_rng(3)
    objs = [rand_bf16(rng, L * 2 * G * nkv * d) for _ in range(n_chunks)]
    table = np.array([7, 2, 9, 0], dtype=np.int32)
    pool = np.zeros(oracle.pool_shape(L, P, nkv, Ps, d), dtype=np.uint16)
    for layer in range(L):
        staging = oracle.assemble_layer([o.view(np.uint8) for o in objs], 2 * G * nkv * d * 2, layer)
        oracle.ingest_layer(staging, n_chunks, G, nkv, d, Ps, table, pool, layer)
        k, v = oracle.logical_kv(objs, G, nkv, d, layer)
        for T in range(n_chunks * G):
            page, slot = table[T // Ps], T % Ps
            for h in range(nkv):
                blk_k = pool[layer, 0, page, h].reshape(Ps, d)
                blk_v = pool[layer, 1, page, h].reshape(Ps, d)
                assert np.array_equal(blk_k[slot], k[T, h])
                assert np.array_equal(blk_v[slot], v[T, h])


def test_ingest_copies_nan_and_denormal_bits():
    G = Ps = 16
    nkv, d = 1, 8
    staging = np.array([0x7FC1, 0xFF80, 0x0001, 0x8001, 0x7F80, 0xFFFF, 0x0000, 0x8000] * (2 * G),
                       dtype=np.uint16)
    pool = np.zeros(oracle.pool_shape(1, 2, nkv, Ps, d), dtype=np.uint16)
    oracle.ingest_layer(staging, 1, G, nkv, d, Ps, np.array([1], np.int32), pool, 0)
    back = oracle.gather_layer(pool, 0, np.array([1], np.int32), 1, G, nkv, d, Ps)
    assert np.array_equal(back, staging)


def test_ingest_rejects_out_of_range_page():
    pool = np.zeros(oracle.pool_shape(1, 4, 1, 16, 8), dtype=np.uint16)
    for threads in (1, 2):
        with pytest.raises(ValueError):
            oracle.ingest_layer(np.zeros(2 * 2 * 16 * 8, np.uint16), 2, 16, 1, 8, 16,
                                np.array([1, 4], np.int32), pool, 0, threads=threads)


# ---------------------------------------------------------------------------
# write path: suffix append and chunk-object offload (Section 3 opening:
# the prefill node materialises the full KV state; new chunks go back to
# object storage)
# ---------------------------------------------------------------------------

def _no_sentinel(rng, shape):
    x = rand_bf16(rng, shape)
    x[x == SENTINEL] = 0
    return x


def test_append_puts_each_suffix_token_where_paging_says():
    # prefix of 40 tokens: the suffix starts mid-page (page 2, slot 8)
    L, nkv, d, Ps, P, layer, Tp, Ts = 2, 2, 8, 16, 12, 1, 40, 29
    rng = np.random.default_rng(11)
    k, v = _no_sentinel(rng, (Ts, nkv, d)), _no_sentinel(rng, (Ts, nkv, d))
    table = rng.permutation(P)[:-(-(Tp + Ts) // Ps)].astype(np.int32)
    pool = np.full(oracle.pool_shape(L, P, nkv, Ps, d), SENTINEL, dtype=np.uint16)
    oracle.append_suffix(k, v, Tp, table, pool, layer, Ps)
    for i in range(Ts):
        T = Tp + i
        page, slot = table[T // Ps], T % Ps
        for h in range(nkv):
            assert np.array_equal(pool[layer, 0, page, h].reshape(Ps, d)[slot], k[i, h])
            assert np.array_equal(pool[layer, 1, page, h].reshape(Ps, d)[slot], v[i, h])
    # exactly the suffix rows were written: nothing of the prefix, no other layer
    assert (pool != SENTINEL).sum() == 2 * Ts * nkv * d
    assert (pool[0] == SENTINEL).all()
    first = pool[layer, :, table[Tp // Ps]].reshape(2, nkv, Ps, d)
    assert (first[:, :, :Tp % Ps] == SENTINEL).all()


def test_append_rejects_a_table_too_short_for_the_suffix():
    pool = np.zeros(oracle.pool_shape(1, 4, 1, 16, 8), dtype=np.uint16)
    kv = np.zeros((9, 1, 8), np.uint16)
    with pytest.raises(ValueError):       # tokens 8..16 need a second page
        oracle.append_suffix(kv, kv, 8, np.array([2], np.int32), pool, 0, 16)


@pytest.mark.parametrize("G,Ps", [(32, 16), (16, 16), (8, 16)])
def test_chunk_gather_inverts_the_scatter_of_every_layer(G, Ps):
    L, nkv, d, N, P = 3, 2, 8, 5, 24
    rng = np.random.default_rng(G)
    objs = np.stack([rand_bf16(rng, L * 2 * G * nkv * d) for _ in range(N)])
    table = rng.permutation(P)[:-(-N * G // Ps)].astype(np.int32)
    pool = np.zeros(oracle.pool_shape(L, P, nkv, Ps, d), dtype=np.uint16)
    for layer in range(L):
        staging = oracle.assemble_layer([o.view(np.uint8) for o in objs], 2 * G * nkv * d * 2, layer)
        oracle.ingest_layer(staging, N, G, nkv, d, Ps, table, pool, layer)
    assert np.array_equal(oracle.gather_chunks(pool, table, 0, N, G, nkv, d, Ps), objs)
    assert np.array_equal(oracle.gather_chunks(pool, table, 1, 2, G, nkv, d, Ps), objs[1:3])
    assert oracle.gather_chunks(pool, table, 2, 0, G, nkv, d, Ps).shape == (0, L * 2 * G * nkv * d)


def test_append_then_offload_gives_the_suffix_chunk_objects():
    # two prefix chunks, three suffix chunks of G tokens: after the append the
    # pool holds the full KV state; offloading chunks 2..4 must give objects
    # whose layer l is K then V of that chunk's suffix tokens (KV_L2TD),
    # assembled here by plain concatenation
    L, nkv, d, G, Ps, P = 2, 2, 8, 32, 16, 16
    n_pre, n_suf = 2, 3
    Tp, Ts = n_pre * G, n_suf * G
    rng = np.random.default_rng(5)
    pre = np.stack([rand_bf16(rng, L * 2 * G * nkv * d) for _ in range(n_pre)])
    k = [rand_bf16(rng, (Ts, nkv, d)) for _ in range(L)]
    v = [rand_bf16(rng, (Ts, nkv, d)) for _ in range(L)]
    table = rng.permutation(P)[:(Tp + Ts) // Ps].astype(np.int32)
    pool = np.zeros(oracle.pool_shape(L, P, nkv, Ps, d), dtype=np.uint16)
    for layer in range(L):
        staging = oracle.assemble_layer([o.view(np.uint8) for o in pre], 2 * G * nkv * d * 2, layer)
        oracle.ingest_layer(staging, n_pre, G, nkv, d, Ps, table, pool, layer)
        oracle.append_suffix(k[layer], v[layer], Tp, table, pool, layer, Ps)
    want = np.stack([np.concatenate([np.concatenate([k[l][s * G:(s + 1) * G].ravel(),
                                                     v[l][s * G:(s + 1) * G].ravel()]) for l in range(L)])
                     for s in range(n_suf)])
    assert np.array_equal(oracle.gather_chunks(pool, table, n_pre, n_suf, G, nkv, d, Ps), want)
    assert np.array_equal(oracle.gather_chunks(pool, table, 0, n_pre, G, nkv, d, Ps), pre)


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------

def _sdpa_reference(q, kp, vp, kn, vn):
    """float64 torch scaled_dot_product_attention (library routine) with GQA
    by repeating KV heads and an explicit boolean mask."""
    Ts, nq, d = q.shape
    Tp, nkv = kp.shape[0], kn.shape[1]
    K = torch.from_numpy(np.concatenate([f64(kp), f64(kn)], 0))      # [Tp+Ts][nkv][d]
    V = torch.from_numpy(np.concatenate([f64(vp), f64(vn)], 0))
    Q = torch.from_numpy(f64(q))
    grp = nq // nkv
    K = K.repeat_interleave(grp, dim=1).permute(1, 0, 2)              # [nq][T][d]
    V = V.repeat_interleave(grp, dim=1).permute(1, 0, 2)
    Q = Q.permute(1, 0, 2)
    mask = torch.ones(Ts, Tp + Ts, dtype=torch.bool)
    mask[:, Tp:] = torch.tril(torch.ones(Ts, Ts, dtype=torch.bool))
    out = torch.nn.functional.scaled_dot_product_attention(Q, K, V, attn_mask=mask)
    return out.permute(1, 0, 2).numpy()


def _inputs(rng, Tp, Ts, nq, nkv, d, scale=1.0):
    return (rand_bf16(rng, (Ts, nq, d), scale), rand_bf16(rng, (Tp, nkv, d)), rand_bf16(rng, (Tp, nkv, d)),
            rand_bf16(rng, (Ts, nkv, d)), rand_bf16(rng, (Ts, nkv, d)))


@pytest.mark.parametrize("Tp,Ts,nq,nkv,d", [
    (256, 32, 4, 2, 64),     # the tiny workload's shape
    (0, 5, 4, 4, 16),        # no cached prefix, MHA
    (37, 1, 8, 1, 32),       # ragged prefix, one suffix token, 8-way GQA
    (48, 17, 6, 2, 8),
])
def test_attention_matches_sdpa(Tp, Ts, nq, nkv, d):
    rng = np.random.default_rng(Tp * 131 + Ts)
    q, kp, vp, kn, vn = _inputs(rng, Tp, Ts, nq, nkv, d, scale=2.0)
    got = oracle.attention(q, kp, vp, kn, vn)
    ref = _sdpa_reference(q, kp, vp, kn, vn)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-12)


def test_attention_row_subset_equals_full():
    rng = np.random.default_rng(11)
    q, kp, vp, kn, vn = _inputs(rng, 40, 9, 4, 2, 16)
    full = oracle.attention(q, kp, vp, kn, vn)
    rows = [8, 0, 3]
    sub = oracle.attention(q, kp, vp, kn, vn, rows=rows)
    assert np.array_equal(sub, full[rows])


def test_constant_values_give_that_constant():
    rng = np.random.default_rng(5)
    Tp, Ts, nq, nkv, d = 30, 6, 4, 2, 16
    q, kp, _, kn, _ = _inputs(rng, Tp, Ts, nq, nkv, d, scale=3.0)
    c = kvgen.f32_to_bf16_bits(rng.standard_normal(d).astype(np.float32))
    vp = np.broadcast_to(c, (Tp, nkv, d)).copy()
    vn = np.broadcast_to(c, (Ts, nkv, d)).copy()
    got = oracle.attention(q, kp, vp, kn, vn)
    np.testing.assert_allclose(got, np.broadcast_to(f64(c), got.shape), rtol=0, atol=1e-14)


def test_equal_keys_average_the_visible_values():
    # identical keys -> uniform weights -> mean of the Tp + i + 1 visible value rows
    rng = np.random.default_rng(6)
    Tp, Ts, nq, nkv, d = 21, 7, 4, 2, 8
    q, _, vp, _, vn = _inputs(rng, Tp, Ts, nq, nkv, d)
    krow = kvgen.f32_to_bf16_bits(rng.standard_normal((1, nkv, d)).astype(np.float32))
    kp = np.repeat(krow, Tp, 0)
    kn = np.repeat(krow, Ts, 0)
    got = oracle.attention(q, kp, vp, kn, vn)
    V = np.concatenate([f64(vp), f64(vn)], 0)
    for i in range(Ts):
        for h in range(nq):
            g = h // (nq // nkv)
            np.testing.assert_allclose(got[i, h], V[:Tp + i + 1, g].mean(0), rtol=1e-12, atol=1e-13)


def test_single_token_without_prefix_returns_its_value():
    rng = np.random.default_rng(8)
    q, kp, vp, kn, vn = _inputs(rng, 0, 1, 4, 2, 16)
    got = oracle.attention(q, kp, vp, kn, vn)
    for h in range(4):
        assert np.array_equal(got[0, h], f64(vn[0, h // 2]))


def test_dominant_logit_selects_that_value_row():
    # one-hot keys; q points at key j* with a large weight -> output is v_{j*}
    Tp, Ts, nq, nkv, d = 24, 4, 2, 1, 32
    rng = np.random.default_rng(9)
    one = kvgen.f32_to_bf16_bits(np.float32([1.0]))[0]
    big = kvgen.f32_to_bf16_bits(np.float32([400.0]))[0]
    kp = np.zeros((Tp, nkv, d), np.uint16)
    kn = np.zeros((Ts, nkv, d), np.uint16)
    for j in range(Tp):
        kp[j, 0, j % d] = one
    for j in range(Ts):
        kn[j, 0, (Tp + j) % d] = one
    vp, vn = rand_bf16(rng, (Tp, nkv, d)), rand_bf16(rng, (Ts, nkv, d))
    q = np.zeros((Ts, nq, d), np.uint16)
    target = [3, 17, 0, 11]
    for i, j in enumerate(target):
        q[i, :, j] = big
    got = oracle.attention(q, kp, vp, kn, vn)
    for i, j in enumerate(target):
        np.testing.assert_allclose(got[i], np.broadcast_to(f64(vp[j, 0]), (nq, d)), atol=1e-15)


def _numpy_causal_attention(Q, K, V):
    """Plain causal softmax attention over one whole sequence (MHA), float64."""
    T, d = Q.shape
    S = Q @ K.T / math.sqrt(d)
    S[np.triu_indices(T, 1)] = -np.inf
    S -= S.max(1, keepdims=True)
    W = np.exp(S)
    return (W / W.sum(1, keepdims=True)) @ V


def test_prefix_cached_equals_full_recompute():
    # attention of the suffix over a cached prefix equals the suffix rows of
    # ordinary causal attention over the concatenated sequence
    rng = np.random.default_rng(10)
    Tp, Ts, nq, nkv, d = 33, 11, 6, 3, 16
    grp = nq // nkv
    q, kp, vp, kn, vn = _inputs(rng, Tp, Ts, nq, nkv, d)
    q_prefix = rand_bf16(rng, (Tp, nq, d))          # queries of the cached part (discarded)
    got = oracle.attention(q, kp, vp, kn, vn)
    Qall = np.concatenate([f64(q_prefix), f64(q)], 0)
    Kall = np.concatenate([f64(kp), f64(kn)], 0)
    Vall = np.concatenate([f64(vp), f64(vn)], 0)
    for h in range(nq):
        full = _numpy_causal_attention(Qall[:, h], Kall[:, h // grp], Vall[:, h // grp])
        np.testing.assert_allclose(got[:, h], full[Tp:], rtol=1e-12, atol=1e-13)


def test_generator_chunk_objects_are_the_layer_slices():
    # the generator's object j, layer l equals the (seed, req, l) stream row j
    objs = kvgen.chunk_objects(3, 0, 4, 6, 32, threads=3)
    for layer in range(4):
        assert np.array_equal(objs[:, layer], kvgen.chunk_layer_slices(3, 0, layer, 6, 32))
    vals = kvgen.bf16_bits_to_f32(objs)
    assert abs(float(vals.mean())) < 0.1 and abs(float(vals.std()) - 1) < 0.1


def test_generator_block_tables_distinct_and_interleaved():
    tables = kvgen.block_tables(4, [5, 3, 7], 60)
    allp = np.concatenate(tables)
    assert np.unique(allp).size == allp.size == 15
    assert all((t >= 0).all() and (t < 60).all() for t in tables)
    assert [len(t) for t in tables] == [5, 3, 7]


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -2.5, np.inf], dtype=np.float32)
    b = kvgen.f32_to_bf16_bits(x)
    # 1+2^-8 is a tie between 1 and 1+2^-7 -> even (1.0); 1+3*2^-8 -> 1+2^-6... (ties to even)
    assert kvgen.bf16_bits_to_f32(b).tolist() == [1.0, 1.0, 1.0 + 2 ** -6, -2.5, np.inf]
