"""GPU parity of the rest-of-layer compute window (O, gate/up, SiLU gating,
down, next layer's QKV) against the float64 oracle, stage by stage; the
pipeline with the window after every attention; and per-stream workspaces
when requests compute on streams of their own."""
import zlib

import numpy as np
import pytest

import kvgen
from oracle import layer as olayer
from tests.gpu_util import RequestSet, assert_attention_close, from_dev, require_gpu, to_dev

pytestmark = pytest.mark.gpu

# |got - ref| <= ULPS * 2^-8 * max(|ref|, 1) element-wise (a few bf16 ulps:
# rounding points agree except near ties, and a differing input moves later
# stages by about one ulp), and relative L2 error <= REL_L2
ULPS, REL_L2 = 4.0, 2e-3


@pytest.fixture(autouse=True)
def _gpu():
    require_gpu()
    import torch
    torch.cuda.synchronize()
    yield
    torch.cuda.synchronize()


def _weights(seed, L, H, F, NQ):
    """Per-stage stacks [L][K][N] (host uint16) from kvgen."""
    shapes = kvgen.layer_weight_shapes(H, F, NQ)
    return [np.stack([kvgen.layer_weight(seed, i, l, K, N) for l in range(L)]) for i, (K, N) in enumerate(shapes)]


def _device_weights(w_host, F):
    from paper_2605_22850_amd import LayerWeights
    return LayerWeights(F, *(to_dev(w.reshape(-1)) for w in w_host))


def _close(got, ref, what):
    g = olayer.bf16_to_f64(got)
    r = olayer.bf16_to_f64(ref)
    err = np.abs(g - r)
    bound = ULPS * 2.0 ** -8 * np.maximum(np.abs(r), 1.0)
    worst = float((err / bound).max()) if err.size else 0.0
    rel = float(np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-300))
    assert np.isfinite(g).all() and worst <= 1.0 and rel <= REL_L2, \
        f"{what}: worst error {worst:.2f} of the bound, rel L2 {rel:.2e}"
    return rel


# (nq, nkv, d, F, T, L, layer, sampled rows or None)
CASES = {
    "small": (8, 2, 64, 1024, 37, 2, 1, None),
    "one-row": (4, 4, 64, 256, 1, 1, 0, None),
    "gqa-d128": (16, 4, 128, 2816, 200, 2, 1, None),
    "llama8b-layer-512-tokens": (32, 8, 128, 14336, 512, 1, 0, 16),
    # 20000 rows go through the chain in two row blocks (18724 + 1276)
    "llama8b-layer-two-row-blocks": (32, 8, 128, 14336, 20000, 1, 0, 16),
}
ROW_BLOCK_8B = (1 << 29) // (2 * 14336)


@pytest.mark.timeout(300)
@pytest.mark.parametrize("name", list(CASES))
def test_rest_of_layer_matches_oracle(name):
    import torch
    import paper_2605_22850_amd as oc
    nq, nkv, d, F, T, L, lay, n_rows = CASES[name]
    seed = zlib.crc32(name.encode()) & 0xFFFF
    H, NQ = nq * d, (nq + 2 * nkv) * d
    print(f"[layer] {name}: H={H} F={F} T={T}", flush=True)
    layout = oc.Layout(L, nq, nkv, d, 16, 16, 8)
    w_host = _weights(seed, L, H, F, NQ)
    w = _device_weights(w_host, F)
    attn = kvgen.suffix_tensor(seed, kvgen.KIND_ACT, 0, lay, (T, H))
    cols = {"o": H, "gu": 2 * F, "act": F, "h": H, "qkv": NQ}
    bufs = {k: torch.full((T, c), -1, dtype=torch.int16, device="cuda") for k, c in cols.items()}
    oc.oc_rest_of_layer(to_dev(attn), T, layout, w, lay, bufs["o"], bufs["gu"], bufs["act"], bufs["h"], bufs["qkv"])
    torch.cuda.synchronize()
    rows = np.arange(T) if n_rows is None else np.unique(np.r_[0, T - 1, np.random.default_rng(seed).choice(
        T, n_rows - 2, replace=False)])
    if T > ROW_BLOCK_8B:
        rows = np.unique(np.r_[rows, ROW_BLOCK_8B - 1, ROW_BLOCK_8B])     # both sides of the block edge
    ref = olayer.rest_of_layer(attn[rows], *(m[lay] for m in w_host))
    for k in cols:
        rel = _close(from_dev(bufs[k])[rows], ref[k], f"{name} stage {k}")
        print(f"  {k}: rel L2 {rel:.2e}", flush=True)


def _run(rs, mode, **kw):
    import paper_2605_22850_amd as oc
    ctx = rs.context(mode, **kw)
    try:
        return oc.oc_pipeline_run(ctx, rs.reqs, rs.L)
    finally:
        oc.oc_context_destroy(ctx)


def test_pipeline_runs_the_window_after_every_attention():
    import paper_2605_22850_amd as oc
    print("[layer] pipeline with the rest of the layer", flush=True)
    L, nq, nkv, d, F = 3, 8, 2, 128, 2048
    rs = RequestSet(L, nq, nkv, d, [256, 128], [40, 70], 96, seed=6).upload(with_payload=True)
    w = _device_weights(_weights(6, L, nq * d, F, (nq + 2 * nkv) * d), F)
    _run(rs, oc.OC_MODE_DEVICE_STAGED)
    base = [from_dev(r.out) for r in rs.reqs]
    for name, mode in (("hbm", oc.OC_MODE_HBM_RESIDENT), ("staged", oc.OC_MODE_DEVICE_STAGED),
                       ("producer", oc.OC_MODE_PRODUCER)):
        for r in rs.reqs:
            r.out.zero_()
        _run(rs, mode, layer_weights=w)
        for r, req in enumerate(rs.reqs):
            assert np.array_equal(from_dev(req.out), base[r]), f"{name}: request {r} output changed"

    # the window makes every layer's compute longer: warm HBM-resident runs,
    # where done - ingested is exactly the layer's compute
    def layer_ms(**kw):
        _run(rs, oc.OC_MODE_HBM_RESIDENT, **kw)
        stats = _run(rs, oc.OC_MODE_HBM_RESIDENT, **kw)
        return np.median([s["done_ms"][l] - s["ingested_ms"][l] for s in stats for l in range(L)])
    c_base, c_with = layer_ms(), layer_ms(layer_weights=w)
    assert c_with > c_base, (c_with, c_base)
    for r in range(2):
        assert_attention_close(base[r][L - 1], rs.expected_out(r, L - 1), f"request {r}")
    bad = oc.LayerWeights(100, w.w_o, w.w_gate_up, w.w_down, w.w_qkv)
    with pytest.raises(oc.OcError):
        _run(rs, oc.OC_MODE_DEVICE_STAGED, layer_weights=bad)


def test_requests_on_their_own_streams_do_not_share_a_workspace():
    # with emulated windows each request's attention runs on a stream of its
    # own and the attentions overlap; their split-KV partials (every request
    # here splits its keys) must not collide
    import paper_2605_22850_amd as oc
    print("[layer] overlapping requests, per-stream workspaces", flush=True)
    rs = RequestSet(3, 4, 2, 64, [2048, 1024, 1536], [16, 24, 8], 512, seed=7).upload(with_payload=True)
    _run(rs, oc.OC_MODE_DEVICE_STAGED, attention_per_request=True)
    base = [from_dev(r.out) for r in rs.reqs]
    for r in rs.reqs:
        r.layer_compute_s = 2e-4
    for _ in range(3):
        for r in rs.reqs:
            r.out.zero_()
        _run(rs, oc.OC_MODE_DEVICE_STAGED, emulate_compute=True)
        for r, req in enumerate(rs.reqs):
            assert np.array_equal(from_dev(req.out), base[r]), f"request {r} differs with per-request streams"
