"""Property tests of the oracle over generated shapes: its scatter against
the independent numpy formulation, and its attention against torch's
float64 scaled_dot_product_attention (a library routine), for chunk and
page sizes that divide, fill or straddle each other, empty and ragged
prefixes, GQA groups 1-4 and suffixes of one token up."""
import numpy as np
from hypothesis import HealthCheck, given, settings
from hypothesis import strategies as st

import oracle
from tests.test_oracle import SENTINEL, _inputs, _numpy_scatter, _sdpa_reference

SETTINGS = settings(max_examples=60, deadline=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow])


@SETTINGS
@given(G=st.sampled_from([1, 2, 3, 8, 12, 16, 24, 32]), Ps=st.sampled_from([8, 16, 24, 32]),
       n_chunks=st.integers(0, 6), nkv=st.integers(1, 4), d=st.sampled_from([8, 16, 24]),
       L=st.integers(1, 3), layer_pick=st.integers(0, 2), extra_pages=st.integers(0, 5),
       seed=st.integers(0, 2**31 - 1))
def test_scatter_matches_numpy_and_gather_inverts_it(G, Ps, n_chunks, nkv, d, L, layer_pick, extra_pages, seed):
    rng = np.random.default_rng(seed)
    layer = layer_pick % L
    need = -(-n_chunks * G // Ps)
    P = max(1, need + extra_pages)
    staging = rng.integers(0, 1 << 16, n_chunks * 2 * G * nkv * d, dtype=np.uint16)
    table = rng.permutation(P)[:need].astype(np.int32)
    pool = np.full(oracle.pool_shape(L, P, nkv, Ps, d), SENTINEL, dtype=np.uint16)
    ref = pool.copy()
    oracle.ingest_layer(staging, n_chunks, G, nkv, d, Ps, table, pool, layer)
    _numpy_scatter(staging, n_chunks, G, nkv, d, Ps, table, ref, layer)
    assert np.array_equal(pool, ref)
    # exactly the prefix's rows were written: 2 * T_p rows of d elements
    assert (pool != SENTINEL).sum() <= staging.size
    assert (pool.reshape(L, 2, P, nkv, Ps, d)[[x for x in range(L) if x != layer]] == SENTINEL).all()
    if n_chunks:
        back = oracle.gather_layer(pool, layer, table, n_chunks, G, nkv, d, Ps)
        assert np.array_equal(back, staging)


@SETTINGS
@given(Tp=st.integers(0, 40), Ts=st.integers(1, 12), nkv=st.integers(1, 3), grp=st.integers(1, 4),
       d=st.sampled_from([8, 16]), scale=st.sampled_from([0.5, 1.0, 3.0]), seed=st.integers(0, 2**31 - 1))
def test_attention_matches_library_sdpa(Tp, Ts, nkv, grp, d, scale, seed):
    rng = np.random.default_rng(seed)
    q, kp, vp, kn, vn = _inputs(rng, Tp, Ts, nkv * grp, nkv, d, scale=scale)
    got = oracle.attention(q, kp, vp, kn, vn)
    ref = _sdpa_reference(q, kp, vp, kn, vn)
    np.testing.assert_allclose(got, ref, rtol=1e-11, atol=1e-12)
