"""GPU tests of the layerwise pipeline: every mode reproduces the oracle
(pool bit-exact, attention in tolerance) and the modes agree bit for bit;
slot recycling under a racing producer; several requests sharing a pool and
a rate; pacing and timestamps; injected producer stalls and aborts end in an
error, never a hang; a short payload is caught before it is landed."""
import time

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
        stats = oc.oc_pipeline_run(ctx, rs.reqs, rs.L)
    finally:
        oc.oc_context_destroy(ctx)
    return stats


def _outs(rs):
    return [from_dev(r.out) for r in rs.reqs]


def _prefill_pool_with_layer_calls(rs):
    # HBM-resident baseline: the pool is filled beforehand by per-layer ingest calls
    import torch
    import paper_2605_22850_amd as oc
    from tests.gpu_util import to_dev
    for r, tp in enumerate(rs.prefix):
        for l in range(rs.L):
            st = to_dev(np.ascontiguousarray(rs.objs[r][:, l, :]).reshape(-1))
            oc.oc_kv_layer_ingest(st, tp // rs.G, rs.reqs[r].pages, tp, rs.d_pool, rs.layout, l)
    torch.cuda.synchronize()


def test_modes_match_oracle_and_each_other():
    import paper_2605_22850_amd as oc
    print("[pipeline] tiny, all modes", flush=True)
    rs = RequestSet(2, 4, 2, 64, [256], [32], 64, seed=1).upload(with_payload=True)
    want_pool = rs.expected_pool()
    results = {}
    for name, mode, kw in (("staged", oc.OC_MODE_DEVICE_STAGED, {}),
                           ("producer", oc.OC_MODE_PRODUCER, {}),
                           ("producer-capped", oc.OC_MODE_PRODUCER, {"rate_bytes_per_s": 50e6, "piece_bytes": 16384})):
        rs.d_pool.fill_(np.int16(np.uint16(0x7FC5).view(np.int16)))
        _run(rs, mode, **kw)
        assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), want_pool), name
        results[name] = _outs(rs)
    _prefill_pool_with_layer_calls(rs)
    _run(rs, oc.OC_MODE_HBM_RESIDENT)
    results["hbm"] = _outs(rs)
    for l in range(rs.L):
        assert_attention_close(results["staged"][0][l], rs.expected_out(0, l), f"layer {l}")
    for name in ("producer", "producer-capped", "hbm"):
        assert np.array_equal(results[name][0], results["staged"][0]), name


def test_two_slot_ring_with_racing_producer():
    # an uncapped multi-threaded producer runs as far ahead as two slots let it;
    # any early reuse of a slot would corrupt a layer
    import paper_2605_22850_amd as oc
    print("[pipeline] 2-slot ring", flush=True)
    rs = RequestSet(6, 8, 2, 128, [512], [24], 96, seed=2).upload(with_payload=True)
    _run(rs, oc.OC_MODE_PRODUCER, slots=2, producer_threads=3, piece_bytes=2 * 16 * 2 * 128 * 2)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())
    got = _outs(rs)[0]
    rs.d_pool.zero_()
    _run(rs, oc.OC_MODE_DEVICE_STAGED)
    assert np.array_equal(got, _outs(rs)[0])
    for l in (0, 5):
        assert_attention_close(got[l], rs.expected_out(0, l), f"layer {l}")


def test_run_waits_for_null_stream_work():
    # the 1 GiB pool is refilled 16 times on torch's default stream right
    # before the run, with no synchronisation in between: the run must start
    # after those fills, or they would overwrite pages it has ingested
    import paper_2605_22850_amd as oc
    print("[pipeline] ordering after null-stream work", flush=True)
    rs = RequestSet(2, 4, 2, 64, [256], [32], 65536, seed=3).upload(with_payload=True)
    want = rs.expected_pool()
    ctx = rs.context(oc.OC_MODE_DEVICE_STAGED)
    try:
        fill = np.int16(np.uint16(SENTINEL).view(np.int16))
        for _ in range(16):
            rs.d_pool.fill_(fill)
        oc.oc_pipeline_run(ctx, rs.reqs, rs.L)
    finally:
        oc.oc_context_destroy(ctx)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), want)
    for l in range(rs.L):
        assert_attention_close(from_dev(rs.reqs[0].out)[l], rs.expected_out(0, l), f"layer {l}")


def test_batch_of_requests_sharing_pool_and_rate():
    import paper_2605_22850_amd as oc
    print("[pipeline] 3 requests", flush=True)
    rs = RequestSet(3, 16, 4, 128, [160, 480, 320], [16, 24, 9], 4 * 60, seed=3).upload()
    total = sum(tp * 2 * 4 * 128 * 2 for tp in rs.prefix) * rs.L
    rate = total / 0.05                      # ~50 ms of delivery
    stats = _run(rs, oc.OC_MODE_PRODUCER, rate_bytes_per_s=rate, piece_bytes=65536)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())
    outs = _outs(rs)
    for r in range(3):
        for l in range(rs.L):
            assert_attention_close(outs[r][l], rs.expected_out(r, l), f"request {r} layer {l}")
    # layer-major, request-minor delivery under one shared rate
    last = max(s["ttft_ms"] for s in stats)
    assert last >= 0.95 * total / rate * 1e3


def _rate_set():
    # three requests, per-layer bytes 256 KiB / 512 KiB / 1 MiB, distinct compute windows
    rs = RequestSet(4, 4, 2, 64, [512, 1024, 2048], [16, 16, 16], 512, seed=7).upload(with_payload=True)
    for req, c in zip(rs.reqs, (0.001, 0.020, 0.005)):
        req.layer_compute_s = c
    return rs


def test_allocation_policies_deliver_at_their_rates():
    import paper_2605_22850_amd as oc
    print("[pipeline] allocation policies", flush=True)
    rs = _rate_set()
    want_pool = rs.expected_pool()
    fill = np.int16(np.uint16(SENTINEL).view(np.int16))
    rs.d_pool.fill_(fill)
    # one shared stream (FIFO); one attention launch per request, as the
    # allocation policies run them, so the outputs compare bit for bit
    _run(rs, oc.OC_MODE_PRODUCER, attention_per_request=True)
    ref = _outs(rs)
    for l in range(rs.L):
        for r in range(3):
            assert_attention_close(ref[r][l], rs.expected_out(r, l), f"request {r} layer {l}")
    B = 200e6
    s = [tp * 2 * rs.nkv * rs.d * 2 for tp in rs.prefix]
    c = [req.layer_compute_s for req in rs.reqs]
    for policy in ("equal", "kv_prop", "bw_prop", "stall_opt", "cal_stall_opt"):
        rs.d_pool.fill_(fill)
        for req in rs.reqs:
            req.out.zero_()
        stats = _run(rs, oc.OC_MODE_PRODUCER, rate_bytes_per_s=B, alloc_policy=policy,
                     margin_bytes_per_s=20e6, slots=6)
        assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), want_pool), policy
        assert all(np.array_equal(a, b) for a, b in zip(_outs(rs), ref)), policy
        want = oc.oc_bandwidth_allocate(policy, s, c, B, 20e6)
        for r, st in enumerate(stats):
            assert st["rate_bytes_per_s"] == pytest.approx(want[r], rel=1e-12)
            # request r's last layer cannot be complete before its clock allows,
            # and its own pacing, not the other requests, decides when it is
            t_pace = rs.L * s[r] / want[r] * 1e3
            got = st["produced_ms"][rs.L - 1]
            print(f"  {policy:14s} request {r}: rate {want[r] / 1e6:7.2f} MB/s, last layer produced at "
                  f"{got:7.2f} ms (pacing {t_pace:7.2f} ms)", flush=True)
            assert t_pace * 0.99 <= got <= t_pace * 1.25 + 5.0, (policy, r)


def test_slow_request_does_not_hold_up_a_fast_one():
    # under Equal with a tiny and a large request, the tiny one finishes first
    import paper_2605_22850_amd as oc
    print("[pipeline] per-request progress", flush=True)
    rs = RequestSet(4, 4, 2, 64, [4096, 256], [8, 8], 512, seed=8).upload(with_payload=True)
    stats = _run(rs, oc.OC_MODE_PRODUCER, rate_bytes_per_s=100e6, alloc_policy="equal", slots=2)
    assert stats[1]["ttft_ms"] < 0.25 * stats[0]["ttft_ms"]
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())


def test_allocation_policy_validation():
    import paper_2605_22850_amd as oc
    print("[pipeline] policy validation", flush=True)
    rs = _rate_set()
    with pytest.raises(oc.OcError) as e:
        rs.context(oc.OC_MODE_PRODUCER, alloc_policy="stall_opt")           # no budget
    assert "budget" in str(e.value)
    with pytest.raises(oc.OcError):
        rs.context(oc.OC_MODE_PRODUCER, rate_bytes_per_s=1e8, alloc_policy=9)
    rs.reqs[1].layer_compute_s = 0.0
    with pytest.raises(oc.OcError) as e:
        _run(rs, oc.OC_MODE_PRODUCER, rate_bytes_per_s=1e8, alloc_policy="stall_opt")
    assert "compute" in str(e.value)
    # policies that need no compute windows run without them
    _run(rs, oc.OC_MODE_PRODUCER, rate_bytes_per_s=1e9, alloc_policy="kv_prop")


def test_pacing_and_timestamps():
    import paper_2605_22850_amd as oc
    print("[pipeline] pacing", flush=True)
    rs = RequestSet(4, 8, 2, 128, [1024], [16], 128, seed=4).upload()
    layer_bytes = 1024 * 2 * 2 * 128 * 2
    rate = layer_bytes / 0.010               # 10 ms per layer
    st = _run(rs, oc.OC_MODE_PRODUCER, rate_bytes_per_s=rate, piece_bytes=65536)[0]
    for l in range(rs.L):
        floor_ms = (l + 1) * layer_bytes / rate * 1e3
        assert st["produced_ms"][l] >= floor_ms - 0.5, (l, st["produced_ms"][l], floor_ms)
        assert st["landed_ms"][l] <= st["ingested_ms"][l] <= st["done_ms"][l]
        if l:
            assert st["done_ms"][l - 1] <= st["done_ms"][l]
    assert st["ttft_ms"] >= rs.L * layer_bytes / rate * 1e3 - 0.5
    assert st["ttft_ms"] <= rs.L * layer_bytes / rate * 1e3 + 250.0


def test_injected_stall_times_out_and_context_recovers():
    import paper_2605_22850_amd as oc
    print("[pipeline] stall -> timeout", flush=True)
    rs = RequestSet(3, 8, 2, 128, [256], [8], 32, seed=5).upload()
    ctx = rs.context(oc.OC_MODE_PRODUCER, timeout_ms=300, fault=oc.OC_FAULT_STALL, fault_layer=1)
    try:
        t = time.time()
        with pytest.raises(oc.OcError) as e:
            oc.oc_pipeline_run(ctx, rs.reqs, rs.L)
        assert e.value.status == oc._lib.OC_ETIMEOUT
        assert time.time() - t < 10
        assert "did not arrive" in str(e.value)
    finally:
        oc.oc_context_destroy(ctx)
    _run(rs, oc.OC_MODE_PRODUCER)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())


def test_injected_abort_reports_error():
    import paper_2605_22850_amd as oc
    print("[pipeline] abort", flush=True)
    rs = RequestSet(3, 8, 2, 128, [256], [8], 32, seed=6).upload()
    with pytest.raises(oc.OcError) as e:
        _run(rs, oc.OC_MODE_PRODUCER, fault=oc.OC_FAULT_ABORT, fault_layer=2)
    assert e.value.status == oc._lib.OC_EABORT


def _short_write_rejected(rs, **kw):
    import paper_2605_22850_amd as oc
    with pytest.raises(oc.OcError) as e:
        _run(rs, oc.OC_MODE_PRODUCER, fault=oc.OC_FAULT_SHORT_WRITE, **kw)
    assert e.value.status == oc._lib.OC_ESHORT
    assert "the producer delivered" in str(e.value)
    return str(e.value)


def test_injected_short_write_is_never_landed():
    # layer 1's payload of request 0 ends half a chunk slice early: the run
    # stops before landing it, so layer 0 of every request is in the pool and
    # no later layer was touched; the context's next run is whole
    import paper_2605_22850_amd as oc
    print("[pipeline] short write, layerwise", flush=True)
    rs = RequestSet(4, 8, 2, 128, [256, 160], [8, 5], 64, seed=7).upload()
    S = 2 * rs.G * 2 * 128 * 2
    msg = _short_write_rejected(rs, fault_layer=1, piece_bytes=3 * S)
    assert f"layer 1 of request 0: the producer delivered {16 * S - S // 2} of {16 * S} bytes" in msg
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool(layers=[0]))
    _run(rs, oc.OC_MODE_PRODUCER)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())


def test_injected_short_write_chunkwise_and_paced():
    import paper_2605_22850_amd as oc
    print("[pipeline] short write, chunkwise", flush=True)
    rs = RequestSet(3, 8, 2, 128, [256, 96], [8, 4], 48, seed=8).upload()
    msg = _short_write_rejected(rs, fault_layer=0, delivery="chunkwise")
    assert "chunks 0.." in msg and "of request 0" in msg
    # chunk groups come first and the first one is torn: nothing was landed
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool(layers=[]))
    print("[pipeline] short write, paced by policy", flush=True)
    total = sum(tp * 2 * 2 * 128 * 2 for tp in rs.prefix) * rs.L
    _short_write_rejected(rs, fault_layer=2, alloc_policy="equal", rate_bytes_per_s=total / 0.03,
                          piece_bytes=16384)
    _run(rs, oc.OC_MODE_PRODUCER, alloc_policy="equal", rate_bytes_per_s=total / 0.03, piece_bytes=16384)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())


def test_layer_lands_in_spans_while_produced():
    # 25 MiB layers land in 8 MiB spans as the paced producer's leading
    # pieces complete (3 threads finish pieces out of order; the last piece
    # is ragged), through a ring of two slots, so each slot is refilled and
    # landed again while the next layer's spans are in flight; every layer
    # must reach the pool whole, and a short layer whose first spans were
    # already landed must still never be ingested
    import paper_2605_22850_amd as oc
    print("[pipeline] spans: 25 MiB layers, 256 KiB pieces, 2 slots", flush=True)
    rs = RequestSet(5, 8, 8, 128, [6160], [12], 512, seed=10).upload()
    kw = dict(rate_bytes_per_s=1.0e9, piece_bytes=256 << 10, producer_threads=3, slots=2)
    _run(rs, oc.OC_MODE_PRODUCER, **kw)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())
    out = _outs(rs)[0]
    for l in range(rs.L):
        assert_attention_close(out[l], rs.expected_out(0, l), f"layer {l}")
    rs.d_pool.fill_(np.int16(np.uint16(SENTINEL).view(np.int16)))
    layer = 6160 * 2 * 8 * 128 * 2
    S = 2 * 16 * 8 * 128 * 2
    msg = _short_write_rejected(rs, fault_layer=1, **kw)
    assert f"layer 1 of request 0: the producer delivered {layer - S // 2} of {layer} bytes" in msg
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool(layers=[0]))


def test_two_contexts_run_from_two_threads_at_once():
    # the library from two host threads at the same time, each with its own
    # context and pool: a paced producer (three runs) and device-staged
    # delivery (twenty runs); both pools and every layer's output must come
    # out as when each runs alone
    import threading
    import paper_2605_22850_amd as oc
    print("[pipeline] two contexts, two threads", flush=True)
    a = RequestSet(4, 8, 2, 128, [512, 96], [16, 7], 96, seed=11).upload()
    b = RequestSet(3, 16, 4, 64, [320], [33], 64, seed=12).upload(with_payload=True)
    layer_bytes_a = (512 + 96) * 2 * 2 * 128 * 2
    ctx_a = a.context(oc.OC_MODE_PRODUCER, rate_bytes_per_s=layer_bytes_a * 4 / 0.05, piece_bytes=16384)
    ctx_b = b.context(oc.OC_MODE_DEVICE_STAGED)
    errors = []

    def run(ctx, rs, reps):
        try:
            for _ in range(reps):
                oc.oc_pipeline_run(ctx, rs.reqs, rs.L)
        except Exception as e:          # reported below, from the main thread
            errors.append(e)

    threads = [threading.Thread(target=run, args=(ctx_a, a, 3)), threading.Thread(target=run, args=(ctx_b, b, 20))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=60)
    # a context still in use by a live thread is left alone, not destroyed
    assert not any(t.is_alive() for t in threads), "a pipeline run did not return"
    oc.oc_context_destroy(ctx_a)
    oc.oc_context_destroy(ctx_b)
    assert not errors, errors
    for rs in (a, b):
        assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())
        for r in range(len(rs.reqs)):
            out = from_dev(rs.reqs[r].out)
            for l in range(rs.L):
                assert_attention_close(out[l], rs.expected_out(r, l), f"request {r} layer {l}")


def test_unknown_fault_rejected():
    import paper_2605_22850_amd as oc
    rs = RequestSet(2, 8, 2, 128, [64], [4], 8, seed=9).upload()
    with pytest.raises(oc.OcError) as e:
        rs.context(oc.OC_MODE_PRODUCER, fault=4)
    assert e.value.status == oc._lib.OC_EINVAL


def test_requests_without_a_cached_prefix_through_the_producer():
    # a context made for requests that bring no cached prefix at all
    # (max_prefix_tokens 0) still has its staging ring; every delivery and
    # policy runs, the pool stays untouched and each output is the attention
    # over the suffix alone
    import paper_2605_22850_amd as oc
    print("[pipeline] producer, no cached prefix", flush=True)
    rs = RequestSet(3, 8, 2, 128, [0, 0], [17, 40], 8, seed=13).upload()
    for kw in ({}, {"rate_bytes_per_s": 1e6}, {"delivery": "chunkwise"}, {"delivery": "auto", "theta_bytes": 1e9},
               {"alloc_policy": "equal", "rate_bytes_per_s": 1e6}):
        for r in rs.reqs:
            r.out.zero_()
        _run(rs, oc.OC_MODE_PRODUCER, **kw)
        assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool()), kw
        for r in range(2):
            out = from_dev(rs.reqs[r].out)
            for l in range(rs.L):
                assert_attention_close(out[l], rs.expected_out(r, l), f"{kw} request {r} layer {l}")


def test_bad_request_rejected_before_running():
    import paper_2605_22850_amd as oc
    print("[pipeline] validation", flush=True)
    rs = RequestSet(2, 8, 2, 128, [256], [8], 32, seed=7).upload()
    rs.reqs[0].prefix_tokens = 250          # not a whole number of 16-token chunks
    with pytest.raises(oc.OcError) as e:
        _run(rs, oc.OC_MODE_PRODUCER)
    assert e.value.status == oc._lib.OC_ESHAPE
    assert (from_dev(rs.d_pool) == 0x7FC5).all()


def test_llama8b_4k_capped_pipeline():
    import paper_2605_22850_amd as oc
    print("[pipeline] 8b-4k, 12.5 GB/s", flush=True)
    rs = RequestSet(32, 32, 8, 128, [4096], [128], 1024, seed=2).upload()
    st = _run(rs, oc.OC_MODE_PRODUCER, rate_bytes_per_s=12.5e9)[0]
    total = 4096 * 4096 * 32
    assert st["ttft_ms"] >= total / 12.5e9 * 1e3 * 0.99
    pool = from_dev(rs.d_pool).reshape(rs.pool_shape())
    want = rs.expected_pool(layers=[0, 31])
    for l in (0, 31):
        assert np.array_equal(pool[l], want[l])
    out = _outs(rs)[0]
    rows = [0, 1, 63, 127]
    for l in (0, 31):
        assert_attention_close(out[l][rows], rs.expected_out(0, l, rows=rows), f"layer {l}")
    print(f"  ttft {st['ttft_ms']:.1f} ms (arrival floor {total / 12.5e9 * 1e3:.1f} ms)", flush=True)


def test_emulated_compute_windows_follow_eq3():
    # a stand-in for the rest of the model's per-layer compute: with a window
    # C per layer and a transfer X per layer the run takes eq. (3)'s
    # X_0 + sum max(X, C) + C; two requests' windows overlap on their own
    # streams; the data path is unchanged
    import oracle.model as model
    import paper_2605_22850_amd as oc
    print("[pipeline] emulated compute windows", flush=True)
    rs = RequestSet(4, 4, 2, 64, [256], [16], 64, seed=4).upload(with_payload=True)
    want = rs.expected_pool()
    rs.reqs[0].layer_compute_s = 0.005
    st = _run(rs, oc.OC_MODE_DEVICE_STAGED, emulate_compute=True)[0]
    assert 4 * 5.0 <= st["ttft_ms"] <= 4 * 5.0 + 4.0, st["ttft_ms"]
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), want)
    for l in range(rs.L):
        assert_attention_close(from_dev(rs.reqs[0].out)[l], rs.expected_out(0, l), f"layer {l}")
    # transfer-bound then compute-bound, against eq. (3)
    layer_bytes = 256 * 2 * 2 * 64 * 2
    for x_ms, c_ms in ((8.0, 3.0), (2.0, 6.0)):
        rs.reqs[0].layer_compute_s = c_ms / 1e3
        st = _run(rs, oc.OC_MODE_PRODUCER, emulate_compute=True, rate_bytes_per_s=layer_bytes / (x_ms / 1e3),
                  piece_bytes=4096)[0]
        want_ms = model.layerwise_ttft([x_ms] * 4, [c_ms] * 4)
        assert want_ms * 0.97 <= st["ttft_ms"] <= want_ms * 1.15 + 1.0, (x_ms, c_ms, st["ttft_ms"], want_ms)
    # two requests' windows overlap
    rs2 = RequestSet(4, 4, 2, 64, [256, 128], [16, 8], 64, seed=5).upload(with_payload=True)
    for r in rs2.reqs:
        r.layer_compute_s = 0.005
    stats = _run(rs2, oc.OC_MODE_DEVICE_STAGED, emulate_compute=True)
    assert max(s["ttft_ms"] for s in stats) <= 4 * 5.0 + 6.0, [s["ttft_ms"] for s in stats]
    rs2.reqs[0].layer_compute_s = 11.0
    with pytest.raises(oc.OcError):
        _run(rs2, oc.OC_MODE_DEVICE_STAGED, emulate_compute=True)


# (G, chunks, d): chunk sizes other than the page size; 12 is not a multiple
# of 8 (the per-token decode), and 104, 132 and 168 prefix tokens end inside
# a page
ROWS_KERNEL_CASES = [(8, 13, 64), (12, 11, 128), (24, 7, 128), (64, 3, 128), (256, 2, 128)]


@pytest.mark.timeout(120)
@pytest.mark.parametrize("G,chunks,d", ROWS_KERNEL_CASES)
def test_layerwise_ingest_chunk_sizes(G, chunks, d):
    # every layer after the first of a run is ingested beside the attention
    # by the 8-slot row kernel; the whole pool must equal the oracle's
    # scatter in the device-staged and the producer modes
    import paper_2605_22850_amd as oc
    print(f"[pipeline] G={G} chunks={chunks} d={d}", flush=True)
    rs = RequestSet(3, 8, 2, d, [G * chunks], [24], 64, seed=17, G=G).upload(with_payload=True)
    want_pool = rs.expected_pool()
    for name, mode in (("staged", oc.OC_MODE_DEVICE_STAGED), ("producer", oc.OC_MODE_PRODUCER)):
        rs.d_pool.fill_(np.int16(np.uint16(SENTINEL).view(np.int16)))
        for req in rs.reqs:
            req.out.zero_()
        _run(rs, mode)
        assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), want_pool), f"{name}: pool"
        out = _outs(rs)[0]
        for l in range(rs.L):
            assert_attention_close(out[l], rs.expected_out(0, l), f"{name} G={G} layer {l}")


@pytest.mark.timeout(120)
def test_scheduling_epochs_admit_late_requests_with_released_bandwidth():
    # Section 3.6's epoch rule on the GPU pipeline: two requests share the
    # budget from the start; a third arrives mid-run and is admitted at the
    # first epoch boundary after the short request has finished, with the
    # rate that request released -- the long request's rate never changes.
    # Each request's TTFT (from its arrival) follows eq. (3) at its own rate
    # from its admission; the pool and every output match the oracle.
    import paper_2605_22850_amd as oc
    from oracle import model
    print("[pipeline] scheduling epochs", flush=True)
    L, nq, nkv, d = 4, 8, 2, 64
    pre, suf = [2048, 8192, 4096], [24, 24, 24]
    rs = RequestSet(L, nq, nkv, d, pre, suf, 1024, seed=19).upload(with_payload=True)
    arrival = [0.0, 0.0, 0.02]
    for req, a in zip(rs.reqs, arrival):
        req.arrival_s = a
    B, epoch = 100e6, 0.05
    s = [tp * 2 * nkv * d * 2 for tp in pre]
    want_r, want_t = model.epoch_schedule("equal", s, None, L, arrival, B, epoch=epoch)
    # hand-checked: 50 MB/s each; the short request ends at 4 MiB / 50 MB/s =
    # 84 ms, so the late one is admitted at the 100 ms boundary
    assert want_r == pytest.approx([50e6] * 3) and want_t == pytest.approx([0.0, 0.0, 0.1])
    stats = _run(rs, oc.OC_MODE_PRODUCER, rate_bytes_per_s=B, alloc_policy="equal", epoch_s=epoch, slots=6)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool()), "pool"
    outs = _outs(rs)
    for r in range(3):
        for l in range(L):
            assert_attention_close(outs[r][l], rs.expected_out(r, l), f"request {r} layer {l}")
    for r, st in enumerate(stats):
        assert st["rate_bytes_per_s"] == pytest.approx(want_r[r], rel=1e-12)
        assert st["admitted_ms"] == pytest.approx(want_t[r] * 1e3, abs=1e-9)
        # eq. (3) from the admission, with X = layer bytes / rate and C the
        # measured compute window of each layer; TTFT counts from arrival
        X = [s[r] / want_r[r] * 1e3] * L
        C = [st["done_ms"][l] - max(st["ingested_ms"][l], st["done_ms"][l - 1] if l else 0.0) for l in range(L)]
        model_ms = (want_t[r] - arrival[r]) * 1e3 + model.layerwise_ttft(X, C)
        print(f"  request {r}: admitted {st['admitted_ms']:.1f} ms, ttft {st['ttft_ms']:.2f} ms "
              f"(eq. (3) {model_ms:.2f} ms)", flush=True)
        assert model_ms * 0.99 - 0.5 <= st["ttft_ms"] <= model_ms * 1.05 + 3.0, r
        # no payload of the late request before its admission
        assert min(st["produced_ms"]) >= want_t[r] * 1e3 + X[0] * 0.9


def test_arrivals_need_an_allocation_policy():
    import paper_2605_22850_amd as oc
    rs = RequestSet(2, 4, 2, 64, [256, 256], [8, 8], 64, seed=20).upload(with_payload=True)
    rs.reqs[1].arrival_s = 0.01
    with pytest.raises(oc.OcError) as e:
        _run(rs, oc.OC_MODE_PRODUCER, rate_bytes_per_s=1e8)
    assert "arrival_s" in str(e.value)


def _random_pipeline_cases(n, seed, scheduled=False):
    # seeded pipelines: 1-5 requests (some with no cached prefix) sharing a
    # pool, GQA groups 1-8, d 64/128, chunks of 8-64 tokens, 2-4 layers;
    # device-staged, or the producer with 2-4 slots, 1-4 threads, pieces
    # that do or do not divide into chunk slices, layerwise / chunkwise /
    # eq. (2) delivery, FIFO or an allocation policy (with arrivals during the
    # run and scheduling epochs), capped or not; one launch per layer or per
    # request
    rng = np.random.default_rng(seed)
    cases = []
    while len(cases) < n:
        nkv, grp = int(rng.choice([1, 2, 4, 8])), int(rng.choice([1, 2, 4, 5, 8]))
        d, G, L = int(rng.choice([64, 128])), int(rng.choice([8, 16, 32, 64])), int(rng.integers(2, 5))
        nr = int(rng.integers(1, 6))
        prefix = [0 if rng.random() < 0.15 else G * int(rng.integers(1, 1024 // G + 1)) for _ in range(nr)]
        suffix = [int(rng.integers(1, 80)) for _ in range(nr)]
        if sum(4 * nkv * grp * d * ts * (tp + ts) for tp, ts in zip(prefix, suffix)) * L > 2e9:
            continue
        need = sum(-(-tp // 16) for tp in prefix)
        P = need + int(rng.integers(1, need + 8))
        b = 2 * nkv * d * 2
        kw = {"attention_per_request": bool(rng.random() < 0.3)}
        if scheduled and nr < 2:
            continue
        if rng.random() < 0.3 and not scheduled:
            mode = "staged"
        else:
            mode = "producer"
            kw.update(slots=int(rng.integers(2, 5)), producer_threads=int(rng.integers(1, 5)),
                      piece_bytes=int(2 * G * b * int(rng.integers(1, 5)) + (0 if rng.random() < 0.5 else 1000)))
            delivery = "layerwise" if scheduled else str(rng.choice(["layerwise", "layerwise", "chunkwise", "auto"]))
            policy = (str(rng.choice(["equal", "kv_prop"])) if scheduled else
                      str(rng.choice(["fifo", "equal", "kv_prop"])) if delivery == "layerwise" else "fifo")
            total = max(1, sum(prefix) * b * L)
            rate = 0.0 if policy == "fifo" and rng.random() < 0.4 else total / float(rng.uniform(0.01, 0.04))
            kw.update(delivery=delivery, alloc_policy=policy, rate_bytes_per_s=rate)
            if delivery == "auto":
                kw["theta_bytes"] = float(rng.choice(prefix)) * b * L + 1.0
            if scheduled:
                # requests arriving during the run, admitted by scheduling epochs
                kw["epoch_s"] = float(rng.choice([0.0, 0.004]))
                kw["arrivals"] = [0.0] + [float(rng.uniform(0.0, 0.02)) for _ in range(nr - 1)]
        cases.append((L, nkv * grp, nkv, d, prefix, suffix, P, G, mode, kw))
    return cases


RANDOM_PIPELINES = _random_pipeline_cases(16, 2605) + _random_pipeline_cases(8, 2606, scheduled=True)


@pytest.mark.parametrize("i", range(len(RANDOM_PIPELINES)))
def test_random_pipelines_match_oracle(i):
    import paper_2605_22850_amd as oc
    L, nq, nkv, d, prefix, suffix, P, G, mode, kw = RANDOM_PIPELINES[i]
    print(f"[pipeline random {i}] L {L} nq {nq} nkv {nkv} d {d} G {G} prefix {prefix} suffix {suffix} P {P} "
          f"{mode} {kw}", flush=True)
    rs = RequestSet(L, nq, nkv, d, prefix, suffix, P, seed=200 + i, G=G).upload(with_payload=mode == "staged")
    kw = dict(kw)
    for req, a in zip(rs.reqs, kw.pop("arrivals", [])):
        req.arrival_s = a
    _run(rs, oc.OC_MODE_DEVICE_STAGED if mode == "staged" else oc.OC_MODE_PRODUCER, **kw)
    assert np.array_equal(from_dev(rs.d_pool).reshape(rs.pool_shape()), rs.expected_pool())
    for r in range(len(prefix)):
        out = from_dev(rs.reqs[r].out)
        for l in range(L):
            assert_attention_close(out[l], rs.expected_out(r, l), f"request {r} layer {l}")
