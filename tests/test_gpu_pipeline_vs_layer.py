"""A pipeline run computes the same attention as the single-layer entry point
called layer by layer: key splits, their merge and the per-stream workspace
slices leave no trace in the outputs, which agree bit for bit, run after run,
and match the oracle."""
import numpy as np
import pytest

from tests.gpu_util import RequestSet, assert_attention_close, from_dev, require_gpu

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
    _run(rs, oc.OC_MODE_DEVICE_STAGED)
    first = [from_dev(r.out) for r in rs.reqs]
    for _ in range(2):            # again, from the filled pool
        for req in rs.reqs:
            req.out.zero_()
        _run(rs, oc.OC_MODE_HBM_RESIDENT)
        for r, req in enumerate(rs.reqs):
            assert np.array_equal(from_dev(req.out), first[r]), f"request {r}: second run differs"
    for r in range(len(pre)):
        assert np.array_equal(_single_layer_outputs(rs, r), first[r]), \
            f"request {r}: pipeline and single-layer calls differ"
    rows = [0, suf[0] - 1]
    assert_attention_close(first[0][L - 1][rows], rs.expected_out(0, L - 1, rows=rows), name)
