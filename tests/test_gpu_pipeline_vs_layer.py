"""With one attention launch per request, a pipeline run computes the same
attention as the single-layer entry point called layer by layer: key
splits, their merge and the workspace slices leave no trace in the outputs,
which agree bit for bit, run after run, and match the oracle.  With several
requests batched into one launch per layer (the default), every row of every
layer matches the oracle (and the per-request launches) within the attention
tolerance, run after run bit for bit."""
import numpy as np
import pytest

from tests.gpu_util import SENTINEL, RequestSet, assert_attention_close, from_dev, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    import torch
    torch.cuda.synchronize()
    yield
    torch.cuda.synchronize()


def _run(rs, mode, **kw):
    import paper_2605_22850_amd as oc
    ctx = rs.context(mode, **kw)
    try:
        return oc.oc_pipeline_run(ctx, rs.reqs, rs.L)
    finally:
        oc.oc_context_destroy(ctx)


def _single_layer_outputs(rs, r):
    import torch
    import paper_2605_22850_amd as oc
    req = rs.reqs[r]
    tp, ts = rs.prefix[r], rs.suffix[r]
    ws = torch.empty(oc.oc_attention_workspace_bytes(rs.layout, tp, ts), dtype=torch.uint8, device="cuda")
    outs = []
    for l in range(rs.L):
        out = torch.empty((ts, rs.nq, rs.d), dtype=torch.bfloat16, device="cuda")
        oc.oc_suffix_prefill_layer(req.q[l], req.k_new[l], req.v_new[l], ts, rs.d_pool, rs.layout, req.pages, tp, l,
                                   out, ws)
        torch.cuda.synchronize()
        outs.append(from_dev(out))
    return np.stack(outs)


# (L, nq, nkv, d, prefixes, suffixes, pool pages): every request splits its keys
CASES = {
    "8b-4k-two-layers": (2, 32, 8, 128, [4096], [128], 1024),
    "8b-64k-two-layers": (2, 32, 8, 128, [65536], [512], 4608),
    "three-requests-d64": (3, 8, 2, 64, [2048, 512, 1024], [40, 7, 100], 512),
}


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", list(CASES))
def test_pipeline_equals_single_layer_calls(name):
    import paper_2605_22850_amd as oc
    L, nq, nkv, d, pre, suf, P = CASES[name]
    print(f"[pipeline vs layer] {name}", flush=True)
    rs = RequestSet(L, nq, nkv, d, pre, suf, P, seed=11).upload(with_payload=True)
    for r, (tp, ts) in enumerate(zip(pre, suf)):
        plan_splits = oc.oc_attention_workspace_bytes(rs.layout, tp, ts)
        assert plan_splits > 256, "the case must split its keys"
    _run(rs, oc.OC_MODE_DEVICE_STAGED, attention_per_request=True)
    first = [from_dev(r.out) for r in rs.reqs]
    for _ in range(2):            # again, from the filled pool
        for req in rs.reqs:
            req.out.zero_()
        _run(rs, oc.OC_MODE_HBM_RESIDENT, attention_per_request=True)
        for r, req in enumerate(rs.reqs):
            assert np.array_equal(from_dev(req.out), first[r]), f"request {r}: second run differs"
    for r in range(len(pre)):
        assert np.array_equal(_single_layer_outputs(rs, r), first[r]), \
            f"request {r}: pipeline and single-layer calls differ"
    rows = [0, suf[0] - 1]
    assert_attention_close(first[0][L - 1][rows], rs.expected_out(0, L - 1, rows=rows), name)


BATCH_CASES = {
    "batch-of-8-varied": (2, 32, 8, 128, [4096, 1024, 2048, 512, 3072, 1536, 256, 0], [256] * 8, 2048),
    "three-requests-d64": (3, 8, 2, 64, [2048, 512, 1024], [40, 7, 100], 512),
    "sixteen-small": (2, 8, 2, 64, [256 + 16 * i for i in range(16)], [8 + i for i in range(16)], 1024),
}


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", list(BATCH_CASES))
def test_batched_layer_launch(name):
    # one attention launch per layer for all requests: every request matches
    # the oracle and its own per-request launch within the tolerance, and
    # repeated runs are bit-identical
    import paper_2605_22850_amd as oc
    L, nq, nkv, d, pre, suf, P = BATCH_CASES[name]
    print(f"[batched] {name}", flush=True)
    rs = RequestSet(L, nq, nkv, d, pre, suf, P, seed=13).upload(with_payload=True)
    _run(rs, oc.OC_MODE_DEVICE_STAGED, attention_per_request=True)
    single = [from_dev(r.out) for r in rs.reqs]
    runs = []
    want_pool = rs.expected_pool()
    for mode in (oc.OC_MODE_DEVICE_STAGED, oc.OC_MODE_HBM_RESIDENT, oc.OC_MODE_PRODUCER):
        for req in rs.reqs:
            req.out.zero_()
        if mode == oc.OC_MODE_DEVICE_STAGED:
            rs.d_pool.fill_(np.int16(np.uint16(SENTINEL).view(np.int16)))
        stats = _run(rs, mode)
        if mode == oc.OC_MODE_DEVICE_STAGED:
            assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), want_pool), "ingest"
        runs.append([from_dev(r.out) for r in rs.reqs])
        # one launch: every request's layer is done at the same moment
        for l in range(L):
            assert len({st["done_ms"][l] for st in stats}) == 1, l
    for r in range(len(pre)):
        assert np.array_equal(runs[1][r], runs[0][r]) and np.array_equal(runs[2][r], runs[0][r]), f"request {r}"
        for l in range(L):
            # every row and head of every layer against the oracle, and
            # against the request's own launch
            assert_attention_close(runs[0][r][l], rs.expected_out(r, l), f"{name} request {r} layer {l}")
            assert_attention_close(runs[0][r][l], _f64(single[r][l]), f"{name} request {r} layer {l} vs per-request")


def _f64(bits):
    return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


@pytest.mark.timeout(300)
def test_more_requests_than_one_launch_takes():
    # 17 requests, one more than a batched launch holds: the pipeline falls
    # back to one attention launch per request, and every request still
    # matches the oracle on every row of every layer
    import paper_2605_22850_amd as oc
    n = 17
    pre, suf = [128 + 16 * i for i in range(n)], [5 + i for i in range(n)]
    print(f"[batched] {n} requests", flush=True)
    rs = RequestSet(2, 8, 2, 64, pre, suf, 1024, seed=17).upload(with_payload=True)
    stats = _run(rs, oc.OC_MODE_DEVICE_STAGED)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool()), "ingest"
    assert len({st["done_ms"][1] for st in stats}) > 1, "17 requests cannot share one launch"
    for r in range(n):
        out = from_dev(rs.reqs[r].out)
        for l in range(2):
            assert_attention_close(out[l], rs.expected_out(r, l), f"request {r} layer {l}")
