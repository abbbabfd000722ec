"""The allocation-free attention entry point (static per-device workspace)
gives the same output, bit for bit, as oc_suffix_prefill_layer with a
caller-owned workspace, on two calls in a row through the C ABI, the second
with a smaller input; both also match the float64 oracle."""
import numpy as np
import pytest

from tests.gpu_util import LayerCase, assert_attention_close, from_dev, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    import torch
    torch.cuda.synchronize()
    yield
    torch.cuda.synchronize()


def _noalloc(case, stream=None):
    import torch
    import paper_2605_22850_amd as oc
    out = torch.full((case.Ts, case.nq, case.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    oc.oc_suffix_prefill_layer_noalloc(case.d_q, case.d_k, case.d_v, case.Ts, case.d_pool, case.layout, case.d_table,
                                       case.Tp, case.layer, out, stream)
    return out


@pytest.mark.timeout(120)
def test_noalloc_attention_matches_the_workspace_entry_point():
    import torch
    import paper_2605_22850_amd as oc
    # (nq, nkv, d, G, Ps, chunks, Ts, pool pages): an 8B-shaped layer whose
    # keys split over many workgroups, then a smaller one with a ragged suffix
    shapes = [(32, 8, 128, 16, 16, 256, 128, 1024), (8, 2, 64, 16, 16, 37, 45, 128)]
    cases = []
    for i, (nq, nkv, d, G, Ps, n, ts, P) in enumerate(shapes):
        print(f"[noalloc] case {i}: nq={nq} nkv={nkv} d={d} Tp={n * G} Ts={ts}", flush=True)
        c = LayerCase(nq, nkv, d, G, Ps, n, ts, P, L=2, layer=1, seed=31 + i).upload()
        c.run_ingest()
        assert oc.oc_attention_workspace_bytes(c.layout, c.Tp, c.Ts) > 256, "the case must split its keys"
        cases.append(c)
    torch.cuda.synchronize()
    want = [from_dev(c.run_attention()) for c in cases]
    torch.cuda.synchronize()
    side = torch.cuda.Stream()
    for i, c in enumerate(cases):
        # the second call runs on a stream of its own, after the first
        got = _noalloc(c, side if i else None)
        torch.cuda.synchronize()
        got = from_dev(got)
        assert np.array_equal(got, want[i]), f"case {i}: differs from oc_suffix_prefill_layer"
        rows = sorted({0, c.Ts // 2, c.Ts - 1})
        assert_attention_close(got[rows], c.expected_attention(rows=rows), f"case {i}")
