"""GPU parity of the single-layer entry points against the CPU oracle:
ingest bit-exact over the whole pool, attention within max|err| 2e-2 and
relative L2 5e-3, plus the invariants (gather after scatter is the identity,
a permuted block table gives bit-identical attention, cached-prefix attention
equals recomputing the whole sequence)."""
import zlib

import numpy as np
import pytest

from tests.gpu_util import (LayerCase, SENTINEL, assert_attention_close, from_dev, require_gpu, to_dev)

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    import torch
    torch.cuda.synchronize()
    yield
    torch.cuda.synchronize()


# (nq, nkv, d, G, Ps, n_chunks, Ts, P, L, layer)
INGEST_CASES = {
    "tiny": (4, 2, 64, 16, 16, 16, 32, 64, 2, 1),
    "8b-4k-layer": (32, 8, 128, 16, 16, 256, 128, 1024, 2, 0),
    "two-chunks-per-page-ragged": (8, 2, 128, 8, 16, 37, 17, 64, 2, 1),
    "two-pages-per-chunk": (8, 4, 64, 32, 16, 9, 5, 40, 3, 2),
    "one-chunk": (4, 4, 128, 16, 16, 1, 3, 4, 1, 0),
    "70b-layer-slice": (64, 8, 128, 16, 16, 512, 64, 2048, 2, 1),
}


@pytest.mark.parametrize("name", list(INGEST_CASES))
def test_ingest_bit_exact_whole_pool(name):
    import torch
    nq, nkv, d, G, Ps, n, Ts, P, L, layer = INGEST_CASES[name]
    print(f"[ingest] {name}", flush=True)
    c = LayerCase(nq, nkv, d, G, Ps, n, Ts, P, L, layer, seed=zlib.crc32(name.encode()) & 0xFFFF).upload()
    c.run_ingest()
    torch.cuda.synchronize()
    got = from_dev(c.d_pool).reshape(c.pool_shape())
    assert np.array_equal(got, c.expected_pool()), "pool differs from the oracle's scatter"


@pytest.mark.parametrize("name", ["tiny", "two-chunks-per-page-ragged", "8b-4k-layer"])
def test_gather_after_ingest_is_identity(name):
    import torch
    from paper_2605_22850_amd import oc_kv_layer_gather
    nq, nkv, d, G, Ps, n, Ts, P, L, layer = INGEST_CASES[name]
    print(f"[gather] {name}", flush=True)
    c = LayerCase(nq, nkv, d, G, Ps, n, Ts, P, L, layer, seed=5).upload()
    c.run_ingest()
    back = torch.zeros_like(c.d_staging)
    oc_kv_layer_gather(c.d_table, c.Tp, c.d_pool, c.layout, layer, back, n)
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(back), c.staging)


def test_ingest_copies_special_bit_patterns():
    import torch
    print("[ingest] special bits", flush=True)
    c = LayerCase(4, 2, 64, 16, 16, 4, 4, 8, 1, 0, seed=3)
    pats = np.array([0x7FC1, 0xFF80, 0x0001, 0x8001, 0x7F80, 0xFFFF, 0x0000, 0x8000], np.uint16)
    c.staging = np.resize(pats, c.staging.size).astype(np.uint16)
    c.upload(fill=0x1234)
    c.run_ingest()
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(c.d_pool).reshape(c.pool_shape()), c.expected_pool(fill=0x1234))


# (nq, nkv, d, G, Ps, n_chunks, Ts, P, L, layer)
ATTN_CASES = {
    "tiny-l0": (4, 2, 64, 16, 16, 16, 32, 64, 2, 0),
    "tiny-l1": (4, 2, 64, 16, 16, 16, 32, 64, 2, 1),
    "8b-4k": (32, 8, 128, 16, 16, 256, 128, 1024, 2, 1),
    "no-prefix": (8, 2, 128, 16, 16, 0, 40, 8, 1, 0),
    "one-suffix-token": (8, 2, 128, 16, 16, 20, 1, 64, 1, 0),
    "ragged-prefix-nan-slots": (8, 2, 128, 8, 16, 37, 17, 64, 2, 1),
    "mha": (4, 4, 128, 16, 16, 10, 33, 32, 1, 0),
    "gqa8": (64, 8, 128, 16, 16, 64, 64, 128, 1, 0),
    "d64-long-suffix": (6, 3, 64, 16, 16, 5, 130, 16, 1, 0),
    "suffix-spans-tiles": (32, 8, 128, 16, 16, 33, 100, 80, 1, 0),
}


@pytest.mark.parametrize("name", list(ATTN_CASES))
def test_attention_matches_oracle(name):
    import torch
    nq, nkv, d, G, Ps, n, Ts, P, L, layer = ATTN_CASES[name]
    print(f"[attention] {name}", flush=True)
    c = LayerCase(nq, nkv, d, G, Ps, n, Ts, P, L, layer, seed=(zlib.crc32(name.encode()) & 0xFFF) + 1).upload()
    if n:
        c.run_ingest()
    out = c.run_attention()
    torch.cuda.synchronize()
    assert_attention_close(from_dev(out), c.expected_attention(), name)


# the end-to-end cells' long suffixes: no key splitting, hundreds of row tiles
# per KV head, causal masking over most of the keys; sampled rows (always the
# first, the last and both sides of a row-tile edge)
# (nq, nkv, d, n_chunks of 16, Ts, P)
LONG_SUFFIX_CASES = {
    "64k-context-12.5pct-hit": (32, 8, 128, 512, 57344, 1024),
    "64k-context-50pct-hit": (32, 8, 128, 2048, 32768, 4096),
    "4k-context-12.5pct-hit": (32, 8, 128, 32, 3584, 64),
}


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", list(LONG_SUFFIX_CASES))
def test_attention_long_suffix_sampled_rows(name):
    import torch
    nq, nkv, d, n, Ts, P = LONG_SUFFIX_CASES[name]
    print(f"[attention] {name}", flush=True)
    c = LayerCase(nq, nkv, d, 16, 16, n, Ts, P, 1, 0, seed=(zlib.crc32(name.encode()) & 0xFFF) + 1).upload()
    c.run_ingest()
    out = from_dev(c.run_attention())
    torch.cuda.synchronize()
    rng = np.random.default_rng(3)
    tile_tokens = 256 // (nq // nkv)          # suffix tokens per 256-row tile
    rows = sorted(set([0, Ts - 1, tile_tokens - 1, tile_tokens, Ts // 2, *rng.choice(Ts, 11, replace=False)]))
    assert_attention_close(out[rows], c.expected_attention(rows=rows), name)


def test_attention_permuted_table_is_bit_identical():
    import torch
    print("[attention] permuted table", flush=True)
    base = dict(nq=32, nkv=8, d=128, G=16, Ps=16, n_chunks=64, Ts=48, P=256, L=1, layer=0, seed=9)
    a = LayerCase(**base, table=np.arange(64, dtype=np.int32)).upload()
    rng = np.random.default_rng(4)
    b = LayerCase(**base, table=rng.permutation(256)[:64].astype(np.int32)).upload()
    a.run_ingest()
    b.run_ingest()
    oa, ob = a.run_attention(), b.run_attention()
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(oa), from_dev(ob))


def test_cached_prefix_equals_full_recompute():
    # attention of the suffix over the cached (paged) prefix equals the last
    # rows of attending over the whole sequence with no cache at all
    import torch
    from paper_2605_22850_amd import oc_attention_workspace_bytes, oc_suffix_prefill_layer
    print("[attention] cached == recompute", flush=True)
    c = LayerCase(16, 4, 128, 16, 16, 24, 40, 64, 1, 0, seed=12).upload()
    c.run_ingest()
    cached = from_dev(c.run_attention())
    k, v = c.logical_kv()
    Tall = c.Tp + c.Ts
    rng = np.random.default_rng(2)
    import kvgen
    q_pre = kvgen.f32_to_bf16_bits(rng.standard_normal((c.Tp, c.nq, c.d)).astype(np.float32))
    q_all = to_dev(np.concatenate([q_pre, c.q]), "bf16")
    k_all = to_dev(np.concatenate([k, c.k_new]), "bf16")
    v_all = to_dev(np.concatenate([v, c.v_new]), "bf16")
    ws = torch.empty(oc_attention_workspace_bytes(c.layout, 0, Tall), dtype=torch.uint8, device="cuda")
    out = torch.empty((Tall, c.nq, c.d), dtype=torch.bfloat16, device="cuda")
    oc_suffix_prefill_layer(q_all, k_all, v_all, Tall, c.d_pool, c.layout, None, 0, 0, out, ws)
    torch.cuda.synchronize()
    full = from_dev(out)[c.Tp:]
    f = lambda x: (x.astype(np.uint32) << 16).view(np.float32)
    assert np.abs(f(full) - f(cached)).max() <= 2e-2
    assert_attention_close(full, c.expected_attention(), "recompute")


def test_pool_beyond_two_billion_elements():
    # a pool whose K region alone holds more than 2^31 elements (140000 pages
    # of 8 heads x 16 slots x 128 dims, 9.2 GB in all): pages above the 2^31
    # element mark must be written, read back and attended to exactly as low
    # ones, through every kernel that indexes the pool
    import torch
    from paper_2605_22850_amd import oc_kv_layer_gather, oc_kv_suffix_append
    nq, nkv, d, G, Ps, n, Ts, P = 8, 8, 128, 16, 16, 64, 40, 140000
    top = (1 << 31) // (nkv * Ps * d)                 # first page past the 2^31 element mark
    need = -(-(n * G + Ts) // Ps)                     # prefix pages + room for the suffix
    rng = np.random.default_rng(11)
    table = np.concatenate([rng.choice(np.arange(top, P), need // 2 + 1, replace=False),
                            rng.choice(np.arange(0, top), need - need // 2 - 1, replace=False)])
    table = rng.permutation(table).astype(np.int32)
    print(f"[ingest] pool of {P} pages, {int((table >= top).sum())} of {need} pages above 2^31 elements",
          flush=True)
    c = LayerCase(nq, nkv, d, G, Ps, n, Ts, P, 1, 0, seed=11, table=table).upload()
    assert c.d_pool.numel() // 2 > (1 << 31)
    c.run_ingest()
    oc_kv_suffix_append(c.d_k, c.d_v, Ts, c.d_table, c.Tp, c.d_pool, c.layout, 0)
    out = c.run_attention()
    back = torch.zeros_like(c.d_staging)
    oc_kv_layer_gather(c.d_table, c.Tp, c.d_pool, c.layout, 0, back, n)
    torch.cuda.synchronize()
    # the oracle scatters into a compact pool whose page i stands for table[i]
    compact = np.full(oracle_pool_shape(need, nkv, Ps, d), SENTINEL, dtype=np.uint16)
    ident = np.arange(need, dtype=np.int32)
    import oracle
    oracle.ingest_layer(c.staging, n, G, nkv, d, Ps, ident, compact, 0)
    oracle.append_suffix(c.k_new, c.v_new, c.Tp, ident, compact, 0, Ps)
    pool = c.d_pool.view(1, 2, P, nkv * Ps * d)
    got = from_dev(pool[0][:, torch.from_numpy(table.astype(np.int64)).cuda()].contiguous())
    assert np.array_equal(got, compact[0].reshape(2, need, -1)), "pages differ from the oracle's scatter + append"
    untouched = np.setdiff1d(np.array([top - 1, top, top + 1, P - 1]), table)
    rest = from_dev(pool[0][:, torch.from_numpy(untouched.astype(np.int64)).cuda()].contiguous())
    assert (rest == SENTINEL).all(), "a page outside the table was written"
    assert np.array_equal(from_dev(back), c.staging), "gather after scatter is not the identity"
    assert_attention_close(from_dev(out), c.expected_attention(), "attention over the large pool")


def oracle_pool_shape(P, nkv, Ps, d):
    import oracle
    return oracle.pool_shape(1, P, nkv, Ps, d)


def _random_cases(n, seed):
    # seeded shapes across the supported space: GQA groups 1-8 (odd ones
    # too), head_dim 64 / 128, chunk sizes that divide a page, fill it or
    # straddle pages, empty and ragged prefixes, suffixes of 1-299 tokens
    # (several row tiles and a ragged last one), pools with or without free
    # pages, any layer of 1-3; kept to sizes the oracle computes in well
    # under a second
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        nkv = int(rng.choice([1, 2, 4, 8]))
        grp = int(rng.choice([1, 2, 3, 4, 5, 8]))
        nq, d = nkv * grp, int(rng.choice([64, 128]))
        G = int(rng.choice([8, 16, 24, 32, 64]))
        n_chunks = 0 if rng.random() < 0.1 else int(rng.integers(1, 4096 // G + 1))
        Ts = int(rng.integers(1, 300))
        if 4 * nq * d * Ts * (n_chunks * G + Ts) > 3e9:
            continue
        need = -(-n_chunks * G // 16)
        P = max(1, need + (0 if rng.random() < 0.2 else int(rng.integers(1, 2 * need + 4))))
        L = int(rng.integers(1, 4))
        cases.append((nq, nkv, d, G, 16, n_chunks, Ts, P, L, int(rng.integers(0, L))))
    return cases


RANDOM_CASES = _random_cases(40, 2605)


@pytest.mark.parametrize("i", range(len(RANDOM_CASES)))
def test_random_shapes_ingest_and_attention(i):
    # whole pool bit-exact after the ingest, every output row in tolerance
    import torch
    nq, nkv, d, G, Ps, n, Ts, P, L, layer = RANDOM_CASES[i]
    print(f"[random {i}] nq {nq} nkv {nkv} d {d} G {G} chunks {n} Ts {Ts} P {P} L {L} layer {layer}", flush=True)
    c = LayerCase(nq, nkv, d, G, Ps, n, Ts, P, L, layer, seed=100 + i).upload()
    if n:
        c.run_ingest()
    out = c.run_attention()
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(c.d_pool).reshape(c.pool_shape()), c.expected_pool())
    assert_attention_close(from_dev(out), c.expected_attention(), f"random {i}")


# (G, Ps, n_chunks, nkv, d): page sizes other than 16 (any multiple of 8 is a
# valid pool for the data-movement entry points; only the attention needs 16),
# chunks smaller than, equal to, larger than and straddling a page; and head
# sizes the attention does not take (any multiple of 8 moves the same way),
# power-of-two and not, with odd KV-head counts
PAGE_SIZE_CASES = [(8, 8, 23, 2, 64), (16, 8, 11, 8, 128), (24, 8, 7, 2, 128), (8, 24, 29, 2, 64),
                   (16, 24, 13, 8, 128), (48, 24, 5, 4, 64), (16, 32, 17, 8, 128), (8, 32, 31, 1, 64),
                   (64, 32, 4, 2, 128), (40, 48, 6, 8, 128),
                   (16, 16, 9, 3, 96), (16, 16, 7, 2, 256), (32, 16, 5, 5, 32), (8, 16, 13, 1, 8)]


@pytest.mark.parametrize("G,Ps,n,nkv,d", PAGE_SIZE_CASES)
def test_page_sizes_ingest_gather_append(G, Ps, n, nkv, d):
    """Ingest (whole pool bit for bit against the oracle's scatter), the
    gather back into the layer payload, and the suffix append behind the
    prefix (against the oracle's append), for a pool of Ps-slot pages and
    d-element head rows."""
    import torch
    import kvgen
    import oracle
    from paper_2605_22850_amd import oc_kv_layer_gather, oc_kv_suffix_append
    Ts, L, layer = 21, 2, 1
    Tp = n * G
    need = -(-(Tp + Ts) // Ps)
    P = need + 5
    print(f"[page sizes] G {G} Ps {Ps} chunks {n} nkv {nkv} d {d}", flush=True)
    table = kvgen.block_tables(Ps * 1000 + G, [need], P)[0]
    c = LayerCase(2 * nkv, nkv, d, G, Ps, n, Ts, P, L, layer, seed=G * 7 + Ps, table=table).upload()
    c.run_ingest()
    torch.cuda.synchronize()
    want = c.expected_pool()
    assert np.array_equal(from_dev(c.d_pool).reshape(c.pool_shape()), want), "pool differs after the ingest"
    back = torch.zeros_like(c.d_staging)
    oc_kv_layer_gather(c.d_table, Tp, c.d_pool, c.layout, layer, back, n)
    oc_kv_suffix_append(c.d_k, c.d_v, Ts, c.d_table, Tp, c.d_pool, c.layout, layer)
    torch.cuda.synchronize()
    assert np.array_equal(from_dev(back), c.staging), "gather is not the inverse of the ingest"
    oracle.append_suffix(c.k_new, c.v_new, Tp, c.table, want, layer, Ps)
    assert np.array_equal(from_dev(c.d_pool).reshape(c.pool_shape()), want), "pool differs after the append"
