#!/usr/bin/env python3
"""Benchmark of the layerwise prefix-KV hot path on one MI355X.

A step is one pass of the whole path over one batch of requests whose layer
payloads are already in HBM: for every layer, ingest (unpack + scatter into
the paged pool) on the copy stream, then that layer's suffix-prefill
attention on the compute stream once the layer's ingested event has fired --
all layers, two streams, per-layer events.

Reported (one JSON line on stdout):
  value          KV ingest GB/s inside the timed steps: algorithmic bytes
                 (read + write of every layer payload) / summed ingest time,
                 each ingest bracketed by HIP events on the copy stream
  roofline       that ingest against 8 TB/s HBM; traffic = HBM bytes per
                 launch from the committed FETCH_SIZE/WRITE_SIZE summary,
                 null when the kernel source has changed since
  ingest_isolated  the same kernel launched back to back with nothing beside
                 it (kernel capability, not the step); also at the second
                 workload and at tiny (L2-resident, launch-latency bound)
  write_path     offload gather of whole chunk objects, suffix append, and
                 the ingest at 64- and 256-token chunks, each alone
  attention      attention TFLOP/s per layer (HBM-resident pass) against the
                 2.5 PFLOP/s bf16 dense MFMA peak
  ttft_ms        HBM-resident / device-staged / producer uncapped / producer
                 capped at 12.5 GB/s (100 Gbps), mean and std over trials
                 after the first
  added_ttft_ms  capped producer minus HBM-resident, beside the eq. (3) floor
  delivery_sweep layerwise against chunkwise delivery at several producer
                 rates, beside eq. (3) and the chunkwise closed form
  policy_sweep   (--policy-sweep) every bandwidth allocation policy under the
                 shared cap: per-request TTFT and rate beside eq. (3)
  cpu_baseline   the CPU oracle on a bounded sample, on this host

``--zero-kv`` prints a line of its own: HBM-resident runs over an all-zero
pool, then over the ingested N(0,1) pool (same kernels and launch shapes;
the attention's time depends on the K/V values through the chip's clock).

``--profile-summary DB...`` turns rocprofv3 output of this script into the
markdown kept under profiles/ (no GPU needed).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
METRIC = "KV ingest GB/s (%HBM peak); added TTFT vs HBM-resident KV, 4K/64K prefix"
INGEST_SRC = os.path.join(ROOT, "paper_2605_22850_amd", "csrc", "ingest.hip")
CALIB_BYTES = 1 << 30          # plain device-to-device copy used to scale the HBM byte counters
CALIB_COPIES = 3


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def attn_flops(nq, d, tp, ts):
    # QK^T and PV over the unmasked (query, key) pairs
    return 4.0 * nq * d * (ts * tp + ts * (ts + 1) / 2.0)


def mean_std(xs):
    xs = list(xs)
    if not xs:
        return [float("nan"), float("nan")]
    m = sum(xs) / len(xs)
    v = sum((x - m) ** 2 for x in xs) / max(1, len(xs) - 1)
    return [round(m, 4), round(math.sqrt(v), 4)]


def layerwise_floor(X, C):
    # eq. (3): X_0 + sum_{l<L-1} max(X_{l+1}, C_l) + C_{L-1}
    t = X[0]
    for l in range(len(X) - 1):
        t += max(X[l + 1], C[l])
    return t + C[-1]


def file_sha256(path):
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def traffic_file(workload):
    return os.path.join(ROOT, "profiles", f"kv_ingest_kernel_{workload}_hbm_traffic.md")


def read_traffic(workload):
    """HBM bytes per ingest launch from the committed counter summary, or
    None when there is none or the kernel source changed after it was taken."""
    path = traffic_file(workload)
    if not os.path.exists(path):
        return None, "no counter summary"
    text = open(path).read()
    m_b = re.search(r"^traffic_bytes_per_launch:\s*([0-9.eE+]+)", text, re.M)
    m_s = re.search(r"^kernel_source_sha256:\s*([0-9a-f]{64})", text, re.M)
    if not (m_b and m_s):
        return None, "counter summary unreadable"
    if m_s.group(1) != file_sha256(INGEST_SRC):
        return None, "kernel changed since the counters were taken"
    return float(m_b.group(1)), os.path.relpath(path, ROOT)


# ---------------------------------------------------------------------------
# GPU legs
# ---------------------------------------------------------------------------

def setup(wl):
    import torch
    import kvgen
    import paper_2605_22850_amd as oc

    L, nq, nkv, d = wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    layout = oc.Layout(L, nq, nkv, d, wl.page_size, wl.chunk_tokens, wl.pool_pages)
    t = time.time()
    pool = torch.zeros(layout.pool_elems, dtype=torch.int16, device="cuda")
    tables = kvgen.block_tables(wl.seed, [wl.pages_needed(r) for r in range(wl.n_requests)], wl.pool_pages)
    reqs, objs_all = [], []
    b = 2 * nkv * d * 2
    for r in range(wl.n_requests):
        tp, ts = wl.prefix_tokens[r], wl.suffix_tokens[r]
        n = wl.n_chunks(r)
        objs = kvgen.chunk_objects(wl.seed, r, L, n, wl.slice_elems, threads=16)    # [N][L][S/2]
        objs_all.append(objs)
        payload = torch.empty(L * tp * b // 2, dtype=torch.int16, device="cuda")
        for l in range(L):
            lay = np.ascontiguousarray(objs[:, l, :]).reshape(-1).view(np.int16)
            payload[l * tp * b // 2:(l + 1) * tp * b // 2].copy_(torch.from_numpy(lay))
        shape_q, shape_kv = (L, ts, nq, d), (L, ts, nkv, d)

        def suffix(kind, shape):
            a = np.stack([kvgen.suffix_tensor(wl.seed, kind, r, l, shape[1:]) for l in range(L)])
            return torch.from_numpy(a.view(np.int16)).cuda().view(torch.bfloat16)

        reqs.append(oc.Request(tp, ts, torch.from_numpy(tables[r]).cuda(), suffix(kvgen.KIND_Q, shape_q),
                               suffix(kvgen.KIND_KNEW, shape_kv), suffix(kvgen.KIND_VNEW, shape_kv),
                               torch.zeros(shape_q, dtype=torch.bfloat16, device="cuda"),
                               chunk_objects=objs.reshape(n, -1), device_payload=payload))
    torch.cuda.synchronize()
    log(f"[bench] setup {wl.name}: {time.time() - t:.1f} s, pool {pool.numel() * 2 / 2**30:.1f} GiB")
    return layout, pool, reqs, objs_all, tables


RUN_OPTS = {}     # context options every run of this process takes (from the command line)


def run_mode(oc, pool, layout, wl, reqs, mode, trials, **kw):
    ctx = oc.oc_context_create(pool, layout, mode, max(wl.prefix_tokens), max(wl.suffix_tokens),
                               **{**RUN_OPTS, **kw})
    out = []
    try:
        for _ in range(trials):
            st = oc.oc_pipeline_run(ctx, reqs, wl.num_layers)
            out.append((oc.oc_pipeline_last_ms(ctx), st))
    finally:
        oc.oc_context_destroy(ctx)
    return out


def copy_calibration():
    """Plain device-to-device copies of a known size; their byte counters
    scale the ingest kernel's."""
    import torch
    src = torch.ones(CALIB_BYTES // 2, dtype=torch.int16, device="cuda")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(CALIB_COPIES):
        dst.copy_(src)
    torch.cuda.synchronize()
    del src, dst


WARM_S = 0.3     # untimed work before a standalone leg: the clocks leave their idle state


def warm_device(s, one_pass):
    """Untimed work on stream s for at least WARM_S seconds (at least one
    pass).  After an idle stretch (host-side setup, the capped producer
    trials) the first launches run slower while the clocks ramp up."""
    t0 = time.perf_counter()
    while True:
        one_pass()
        s.synchronize()
        if time.perf_counter() - t0 >= WARM_S:
            return


def _sleep_cycles_per_ms(s):
    """Calibrates torch.cuda._sleep (a bounded spin kernel) on stream s."""
    import torch
    with torch.cuda.stream(s):
        a, z = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda._sleep(1000)
        a.record(s)
        torch.cuda._sleep(2_000_000)
        z.record(s)
    s.synchronize()
    return 2_000_000 / max(a.elapsed_time(z), 1e-3)


def gated_passes(s, launches, passes, per_launch=True):
    """Times `passes` passes over `launches` (a list of (enqueue function,
    algorithmic bytes)) on stream s, each launch between two HIP events.
    The events are created before the pass, and the device first spins
    (torch.cuda._sleep) long enough for the host to enqueue the whole pass,
    so that each launch's events measure the device, not the Python host's
    per-call cost.  Returns the per-launch (start, end, bytes) triples and
    one (start, end) pair per pass.  With per_launch False only the pass is
    bracketed (each event marker between launches costs the stream a few
    microseconds)."""
    import torch
    per_ms = _sleep_cycles_per_ms(s)
    evs, spans, host_ms = [], [], 1.0
    with torch.cuda.stream(s):
        for i in range(passes + 1):       # the first pass measures the host's enqueue time only
            pairs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                     for _ in range(len(launches) + 1)]
            for e0, e1 in pairs:          # the device events exist before the timed enqueue
                e0.record(s)
                e1.record(s)
            s.synchronize()
            torch.cuda._sleep(int(per_ms * (2.0 * host_ms + 2.0)))
            t0 = time.perf_counter()
            pairs[-1][0].record(s)
            for (fn, nbytes), (e0, e1) in zip(launches, pairs):
                if not per_launch:
                    fn()
                    continue
                e0.record(s)
                fn()
                e1.record(s)
                if i > 0:
                    evs.append((e0, e1, nbytes))
            pairs[-1][1].record(s)
            host_ms = (time.perf_counter() - t0) * 1e3
            if i > 0:
                spans.append(pairs[-1])
            s.synchronize()
    return evs, spans


def isolated_ingest(oc, wl, layout, pool, reqs, passes):
    """Ingest of every layer of every request, back to back on one stream,
    nothing else running; per-launch HIP events (gated_passes) after
    WARM_S of untimed passes."""
    import torch
    s = torch.cuda.Stream()
    b = 2 * wl.num_kv_heads * wl.head_dim * 2
    launches = []
    for l in range(wl.num_layers):
        for r, rq in enumerate(reqs):
            tp = wl.prefix_tokens[r]
            st = rq.device_payload[l * tp * b // 2:(l + 1) * tp * b // 2]
            launches.append((lambda st=st, rq=rq, tp=tp, l=l:
                             oc.oc_kv_layer_ingest(st, tp // wl.chunk_tokens, rq.pages, tp, pool, layout, l, s),
                             2.0 * tp * b))

    def one_pass():
        for fn, _ in launches:
            fn()
    warm_device(s, one_pass)
    evs, _ = gated_passes(s, launches, passes)
    ms = sum(e0.elapsed_time(e1) for e0, e1, _ in evs)
    nbytes = sum(x for _, _, x in evs)
    gbs = nbytes / (ms / 1e3) / 1e9
    _, spans = gated_passes(s, launches, passes, per_launch=False)
    span_ms = sum(a.elapsed_time(z) for a, z in spans)
    per_launch = nbytes / len(evs)
    size = f"{per_launch / 2**20:.0f} MiB" if per_launch >= 2**20 else f"{per_launch / 2**10:.0f} KiB"
    return {"value": round(gbs, 2), "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4),
            "launches": len(evs), "mean_launch_us": round(ms / len(evs) * 1e3, 3),
            "back_to_back_GBps": round(nbytes / (span_ms / 1e3) / 1e9, 2),
            "how": f"{passes} passes over all {wl.num_layers} layer payloads ({size} read + written per launch) "
                   f"after {WARM_S} s of untimed ones, one stream, nothing beside it; value from HIP events "
                   f"around each launch, back_to_back from passes with one pair of events around the whole "
                   f"pass and none between launches; each pass enqueued before the device starts on it"}


def _rate(evs, how):
    ms = sum(e0.elapsed_time(e1) for e0, e1, _ in evs)
    nbytes = sum(x for _, _, x in evs)
    gbs = nbytes / (ms / 1e3) / 1e9
    return {"value": round(gbs, 2), "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "launches": len(evs),
            "mean_launch_us": round(ms / len(evs) * 1e3, 3), "bytes_per_launch": nbytes / len(evs), "how": how}


def write_path(oc, wl, layout, pool, reqs, passes):
    """The write path and the other chunk sizes, each kernel back to back on
    one stream with nothing beside it, per-launch HIP events (gated_passes):
      offload_gather   every chunk object of each request rebuilt from the
                       pool, all layers in one launch (read + write);
      suffix_append    one layer's suffix K/V appended behind the prefix;
      ingest_g64/g256  the layer ingest with the payload taken as chunks of
                       64 / 256 tokens (the paper's other chunk sizes; the
                       payload bytes are the same, only their order differs).
    Leaves the pool in an unspecified state."""
    import torch
    L, nkv, d, Ps = wl.num_layers, wl.num_kv_heads, wl.head_dim, wl.page_size
    b = 2 * nkv * d * 2
    s = torch.cuda.Stream()
    out = {}
    tp_max = max(wl.prefix_tokens)
    objs = torch.empty(tp_max * b * L // 2, dtype=torch.int16, device="cuda")
    launches = [(lambda rq=rq, tp=tp: oc.oc_kv_chunks_gather(rq.pages, tp, pool, layout, 0, tp // wl.chunk_tokens,
                                                             objs, s), 2.0 * tp * b * L)
                for rq, tp in zip(reqs, wl.prefix_tokens)]
    evs, _ = gated_passes(s, launches, passes)
    del objs
    out["offload_gather"] = _rate(evs, f"{passes} passes; per request one launch over all {L} layers of "
                                       f"its chunk objects (read pool + write objects)")
    # appending needs table room behind the prefix: a table of its own
    tables = [torch.arange(-(-(tp + ts) // Ps), dtype=torch.int32, device="cuda")
              for tp, ts in zip(wl.prefix_tokens, wl.suffix_tokens)]
    launches = [(lambda l=l, r=r, rq=rq: oc.oc_kv_suffix_append(rq.k_new[l], rq.v_new[l], wl.suffix_tokens[r],
                                                                tables[r], wl.prefix_tokens[r], pool, layout, l, s),
                 2.0 * wl.suffix_tokens[r] * b)
                for l in range(L) for r, rq in enumerate(reqs)]
    evs, _ = gated_passes(s, launches, passes)
    out["suffix_append"] = _rate(evs, f"{passes} passes over all {L} layers (read + write of the suffix K/V)")
    for G in (64, 256):
        if any(tp % G for tp in wl.prefix_tokens):
            continue
        lay = oc.Layout(L, wl.num_q_heads, nkv, d, Ps, G, wl.pool_pages)
        launches = []
        for l in range(L):
            for r, rq in enumerate(reqs):
                tp = wl.prefix_tokens[r]
                st = rq.device_payload[l * tp * b // 2:(l + 1) * tp * b // 2]
                launches.append((lambda st=st, rq=rq, tp=tp, l=l, lay=lay:
                                 oc.oc_kv_layer_ingest(st, tp // G, rq.pages, tp, pool, lay, l, s), 2.0 * tp * b))
        evs, _ = gated_passes(s, launches, passes)
        out[f"ingest_g{G}"] = _rate(evs, f"{passes} passes over all {L} layer payloads as {G}-token chunks")
    return out


def ttft_legs(oc, wl, layout, pool, reqs, args, hbm, dev, sweep=True):
    """TTFT of the four modes (HBM-resident and device-staged trials given),
    added TTFT at the cap, the eq. (3) floor and the device-staged gate."""
    L, b = wl.num_layers, 2 * wl.num_kv_heads * wl.head_dim * 2
    trials = max(2, args.trials)
    ttft = {"hbm_resident": mean_std(x[0] for x in hbm[1:]), "device_staged": mean_std(x[0] for x in dev[1:])}
    res = {}
    if not args.no_producer:
        unc = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials, rate_bytes_per_s=0.0)
        log(f"[bench] {wl.name} producer uncapped trials done")
        cap = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials, rate_bytes_per_s=args.cap)
        log(f"[bench] {wl.name} producer capped trials done")
        ttft["producer_uncapped"] = mean_std(x[0] for x in unc[1:])
        ttft["producer_capped"] = mean_std(x[0] for x in cap[1:])
        # eq. (3) floor at the cap: X_l = bytes of layer l / cap, C_l = measured device-staged per-layer time
        layer_bytes = sum(wl.prefix_tokens) * b
        X = [layer_bytes / args.cap * 1e3] * L
        C = [ttft["device_staged"][0] / L] * L
        floor = layerwise_floor(X, C)
        res = {"added_ttft_ms": round(ttft["producer_capped"][0] - ttft["hbm_resident"][0], 3),
               "eq3_floor_ms": round(floor, 3),
               "cap_vs_floor": round(ttft["producer_capped"][0] / floor, 4),
               "arrival_floor_ms": round(L * layer_bytes / args.cap * 1e3, 3)}
    res["gates"] = {"device_staged_over_hbm": round((ttft["device_staged"][0] - ttft["hbm_resident"][0]) /
                                                    ttft["hbm_resident"][0], 4)}
    if not args.no_producer and args.sweep_rates and sweep:
        res["delivery_sweep"] = delivery_sweep(oc, wl, layout, pool, reqs, args, ttft["device_staged"][0] / L)
        sens = bandwidth_sensitivity(res["delivery_sweep"])
        if sens:
            res["bandwidth_sensitivity"] = sens
    return ttft, res


def chunkwise_floor(X, C):
    # Section 3.5's chunkwise baseline: every transfer, then every layer's compute
    return sum(X) + sum(C)


def delivery_sweep(oc, wl, layout, pool, reqs, args, c_layer_ms):
    """Layerwise against chunkwise delivery over a range of producer rates
    (Section 5's bandwidth sensitivity), each beside its model: eq. (3) for
    layerwise, all transfers then all compute for chunkwise, X_l = layer bytes
    / rate, C_l = the measured device-staged time per layer."""
    L, b = wl.num_layers, 2 * wl.num_kv_heads * wl.head_dim * 2
    layer_bytes = sum(wl.prefix_tokens) * b
    out = []
    for gbs in [float(x) for x in args.sweep_rates.split(",")]:
        rate = gbs * 1e9
        trial_s = L * layer_bytes / rate if rate > 0 else 0.0
        if trial_s > args.sweep_max_s:
            out.append({"rate_GBps": gbs, "skipped": f"over {args.sweep_max_s} s per trial"})
            continue
        # rates whose trial takes seconds: one timed trial after the discarded first
        trials = 2 if trial_s > 2.0 else max(2, args.trials // 2)
        row = {"rate_GBps": gbs if rate > 0 else "uncapped", "timed_trials": trials - 1}
        for name in ("layerwise", "chunkwise"):
            runs = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials, rate_bytes_per_s=rate,
                            delivery=name)
            row[f"{name}_ms"] = mean_std(x[0] for x in runs[1:])
        if rate > 0:
            X, C = [layer_bytes / rate * 1e3] * L, [c_layer_ms] * L
            row["eq3_floor_ms"] = round(layerwise_floor(X, C), 3)
            row["chunkwise_floor_ms"] = round(chunkwise_floor(X, C), 3)
        out.append(row)
        log(f"[bench] {wl.name} delivery sweep {gbs} GB/s done")
    return out


def bandwidth_sensitivity(sweep, low=1.25, high=12.5):
    """Relative TTFT increase at `low` GB/s over `high` GB/s (10 over 100
    Gbps: the paper's bandwidth-sensitivity comparison), per delivery."""
    rows = {r["rate_GBps"]: r for r in sweep if "skipped" not in r}
    if low not in rows or high not in rows:
        return None
    return {"rates_GBps": [low, high],
            **{f"{name}_increase": round(rows[low][f"{name}_ms"][0] / rows[high][f"{name}_ms"][0] - 1.0, 4)
               for name in ("layerwise", "chunkwise")}}


POLICIES = ["fifo", "equal", "kv_prop", "bw_prop", "stall_opt", "cal_stall_opt"]


def policy_sweep(oc, wl, layout, pool, reqs, args, hbm):
    """Every bandwidth allocation policy on the workload's requests under one
    shared cap (Section 3.6 and the multi-tenant evaluation): per-request TTFT
    and allocated rate, the eq. (3) prediction at that rate, and the added
    TTFT over an uncapped run (the paper's comparison metric).  Compute
    windows c_i are the measured per-layer attention times of each request."""
    L, b = wl.num_layers, 2 * wl.num_kv_heads * wl.head_dim * 2
    R = len(reqs)
    trials = max(2, args.trials // 2)
    c_ms = [float(np.mean([st[r]["done_ms"][l] - st[r]["ingested_ms"][l] for _, st in hbm[1:] for l in range(L)]))
            for r in range(R)]
    for r, req in enumerate(reqs):
        req.layer_compute_s = c_ms[r] / 1e3
    s_bytes = [wl.prefix_tokens[r] * b for r in range(R)]
    unc = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials, rate_bytes_per_s=0.0)
    base = [float(np.mean([st[r]["ttft_ms"] for _, st in unc[1:]])) for r in range(R)]
    out = {"cap_GBps": args.cap / 1e9, "margin_GBps": args.policy_margin / 1e9,
           "layer_bytes": s_bytes, "compute_ms_per_layer": [round(c, 4) for c in c_ms],
           "uncapped_ttft_ms": [round(t, 3) for t in base], "policies": {}}
    log(f"[bench] policy sweep: uncapped baseline done")
    for pol in POLICIES:
        runs = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials, rate_bytes_per_s=args.cap,
                        alloc_policy=pol, margin_bytes_per_s=args.policy_margin)
        ttft = [float(np.mean([st[r]["ttft_ms"] for _, st in runs[1:]])) for r in range(R)]
        rates = [runs[-1][1][r]["rate_bytes_per_s"] for r in range(R)]
        row = {"ttft_ms": [round(t, 3) for t in ttft], "mean_ttft_ms": round(float(np.mean(ttft)), 3),
               "max_ttft_ms": round(max(ttft), 3),
               "added_ttft_ms": round(float(np.mean([t - u for t, u in zip(ttft, base)])), 3)}
        if pol != "fifo":
            row["rate_GBps"] = [round(x / 1e9, 4) for x in rates]
            # eq. (3) per request at its own rate for the whole run
            row["eq3_ms"] = [round(layerwise_floor([s_bytes[r] / rates[r] * 1e3] * L, [c_ms[r]] * L), 3)
                             if rates[r] > 0 else None for r in range(R)]
        out["policies"][pol] = row
        log(f"[bench] policy sweep: {pol} done")
    eq = out["policies"]["equal"]["added_ttft_ms"]
    for pol in ("stall_opt", "cal_stall_opt"):
        a = out["policies"][pol]["added_ttft_ms"]
        out[f"equal_over_{pol}"] = round(eq / a, 3) if a > 0 else None
    return out


def scheduler_workloads(args):
    """The multi-tenant bandwidth-allocation evaluation: Workloads A/B/C (the
    paper's request cells, cached tokens and A100 compute windows scaled down
    together), every policy under the workload's cap with the per-layer
    compute windows emulated, against an uncapped run.  Reports per-request
    TTFT, allocated rates, eq. (3) per request, and the added TTFT ratio of
    Equal to (Calibrated) Stall-opt -- the paper's headline comparison."""
    # every request computes on a stream of its own; with HIP's default of 4
    # hardware queues per process the streams would share queues and one
    # request's window would hold up the others (must be set before HIP starts)
    os.environ["GPU_MAX_HW_QUEUES"] = "16"
    import torch
    import kvgen
    import paper_2605_22850_amd as oc
    torch.cuda.set_device(0)
    out = {}
    for name in args.scheduler_workloads.split(","):
        wl, windows, cap = kvgen.scheduler_workload(name, scale=args.scheduler_scale)
        layout, pool, reqs, _, _ = setup(wl)
        L, b, R = wl.num_layers, 2 * wl.num_kv_heads * wl.head_dim * 2, wl.n_requests
        for req, w in zip(reqs, windows):
            req.layer_compute_s = w
        s_bytes = [t * b for t in wl.prefix_tokens]
        trials = max(2, args.trials // 2)
        kw = dict(emulate_compute=True, slots=2 * R, piece_bytes=1 << 20)
        unc = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials, rate_bytes_per_s=0.0, **kw)
        base = [float(np.mean([st[r]["ttft_ms"] for _, st in unc[1:]])) for r in range(R)]
        res = {"cap_Gbps": cap * 8 / 1e9, "scale": args.scheduler_scale, "cached_tokens": wl.prefix_tokens,
               "window_ms": [round(w * 1e3, 3) for w in windows], "uncapped_ttft_ms": [round(t, 2) for t in base],
               "policies": {}}
        for pol in POLICIES[1:]:
            runs = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials, rate_bytes_per_s=cap,
                            alloc_policy=pol, margin_bytes_per_s=args.policy_margin, **kw)
            ttft = [float(np.mean([st[r]["ttft_ms"] for _, st in runs[1:]])) for r in range(R)]
            rates = [runs[-1][1][r]["rate_bytes_per_s"] for r in range(R)]
            res["policies"][pol] = {
                "rate_Gbps": [round(x * 8 / 1e9, 2) for x in rates],
                "ttft_ms": [round(t, 2) for t in ttft],
                "eq3_ms": [round(layerwise_floor([s_bytes[r] / rates[r] * 1e3] * L, [windows[r] * 1e3] * L), 2)
                           for r in range(R)],
                "added_ttft_ms": round(float(sum(t - u for t, u in zip(ttft, base))), 2)}
            log(f"[bench] scheduler workload {name}: {pol} done")
        eq = res["policies"]["equal"]["added_ttft_ms"]
        for pol in ("stall_opt", "cal_stall_opt"):
            a = res["policies"][pol]["added_ttft_ms"]
            res[f"equal_over_{pol}"] = round(eq / a, 3) if a > 0 else None
        out[name] = res
        del pool, reqs
        torch.cuda.empty_cache()
    return out


CELLS = [(4096, 0.125), (4096, 0.5), (4096, 0.875), (65536, 0.125), (65536, 0.5), (65536, 0.875)]


def canonical_cells(args):
    """The paper's end-to-end TTFT evaluation shape on this GPU: Llama-3-8B
    (32 layers, 32q/8kv, d 128, FFN 14336) with random weights, contexts of
    4K and 64K tokens at 12.5/50/87.5 % prefix hits stored as G-token chunks;
    every layer computes its attention and the rest of the layer (O,
    gate/up, SiLU, down, QKV GEMMs) on the miss tokens.  Per cell: TTFT with
    the KV HBM-resident, the producer uncapped (host memory over PCIe), and
    capped at 12.5 GB/s layerwise and chunkwise, beside eq. (3) and the
    chunkwise closed form with X_l = layer bytes / cap and C_l measured."""
    import torch
    import kvgen
    import paper_2605_22850_amd as oc
    torch.cuda.set_device(0)
    L, nq, nkv, d, F, Ps, G = 32, 32, 8, 128, 14336, 16, args.cells_chunk
    H, NQ, b = nq * d, (nq + 2 * nkv) * d, 2 * nkv * d * 2
    seed = 8
    gen = torch.Generator(device="cuda")
    gen.manual_seed(seed)

    def randn_bf16(shape, scale=1.0):
        t = torch.empty(shape, dtype=torch.bfloat16, device="cuda")
        flat = t.view(shape[0], -1)
        for i in range(shape[0]):       # one layer at a time: bounded float32 temporaries
            flat[i].copy_(torch.randn(flat.shape[1], generator=gen, device="cuda") * scale)
        return t

    t0 = time.time()
    shapes = kvgen.layer_weight_shapes(H, F, NQ)
    ws = [randn_bf16((L, K, N), K ** -0.5) for K, N in shapes]
    weights = oc.LayerWeights(F, *ws)
    max_tp = max(int(c * r) for c, r in CELLS)
    slice_elems = 2 * G * nkv * d
    objs = kvgen.chunk_objects(seed, 0, L, max_tp // G, slice_elems, threads=16)     # [N][L][S/2]
    log(f"[bench] cells setup: weights {sum(w.numel() for w in ws) * 2 / 2**30:.1f} GiB, "
        f"chunk objects {objs.nbytes / 2**30:.1f} GiB, {time.time() - t0:.1f} s")
    trials = max(2, args.trials // 2)
    out = {"model": "llama-3-8b shape, random weights", "chunk_tokens": G, "cap_GBps": args.cap / 1e9,
           "ffn_dim": F, "cells": []}
    for ctx_len, hit in CELLS:
        tp, ts = int(ctx_len * hit), ctx_len - int(ctx_len * hit)
        n = tp // G
        need = -(-tp // Ps)
        P = 2 * need
        layout = oc.Layout(L, nq, nkv, d, Ps, G, P)
        pool = torch.zeros(layout.pool_elems, dtype=torch.int16, device="cuda")
        table = torch.from_numpy(kvgen.block_tables(seed, [need], P)[0]).cuda()
        q = randn_bf16((L, ts, nq, d))
        kn = randn_bf16((L, ts, nkv, d))
        vn = randn_bf16((L, ts, nkv, d))
        outt = torch.zeros((L, ts, nq, d), dtype=torch.bfloat16, device="cuda")
        reqs = [oc.Request(tp, ts, table, q, kn, vn, outt, chunk_objects=objs[:n].reshape(n, -1))]
        wl = kvgen.Workload(name=f"cell-{ctx_len}-{hit}", num_layers=L, num_q_heads=nq, num_kv_heads=nkv,
                            head_dim=d, page_size=Ps, chunk_tokens=G, prefix_tokens=[tp], suffix_tokens=[ts],
                            pool_pages=P, seed=seed)
        kw = dict(layer_weights=weights)
        res = {"context": ctx_len, "hit": hit, "prefix_tokens": tp, "suffix_tokens": ts}
        # the uncapped producer also fills the pool for the HBM-resident runs
        runs = {"producer_uncapped": run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials,
                                              rate_bytes_per_s=0.0, **kw)}
        runs["hbm_resident"] = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_HBM_RESIDENT, trials, **kw)
        runs["capped_layerwise"] = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials,
                                            rate_bytes_per_s=args.cap, **kw)
        runs["capped_chunkwise"] = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials,
                                            rate_bytes_per_s=args.cap, delivery="chunkwise", **kw)
        ttft = {k: float(np.mean([st[0]["ttft_ms"] for _, st in v[1:]])) for k, v in runs.items()}
        c_ms = [float(np.mean([st[0]["done_ms"][l] - st[0]["ingested_ms"][l] for _, st in runs["hbm_resident"][1:]]))
                for l in range(L)]
        x_ms = [tp * b / args.cap * 1e3] * L
        res["ttft_ms"] = {k: round(v, 2) for k, v in ttft.items()}
        res["compute_ms_per_layer"] = round(float(np.mean(c_ms)), 3)
        res["transfer_ms_per_layer_at_cap"] = round(x_ms[0], 3)
        res["eq3_ms"] = round(layerwise_floor(x_ms, c_ms), 2)
        res["chunkwise_model_ms"] = round(chunkwise_floor(x_ms, c_ms), 2)
        base = ttft["hbm_resident"]
        res["added_over_hbm_pct"] = {k: round((v - base) / base * 100, 2) for k, v in ttft.items()
                                     if k != "hbm_resident"}
        res["capped_layerwise_over_uncapped_pct"] = round(
            (ttft["capped_layerwise"] - ttft["producer_uncapped"]) / ttft["producer_uncapped"] * 100, 2)
        flops = attn_flops(nq, d, tp, ts)
        res["attention_gflop_per_layer"] = round(flops / 1e9, 1)
        res["gemm_gflop_per_layer"] = round(2 * ts * sum(K * N for K, N in shapes) / 1e9, 1)
        res["layer_tflops"] = round((flops + 2 * ts * sum(K * N for K, N in shapes)) / (np.mean(c_ms) / 1e3) / 1e12, 1)
        # the overlap requirement of Section 5.3: the rate at which a layer's
        # transfer takes exactly its compute window
        res["required_GBps"] = round(tp * b / (np.mean(c_ms) / 1e3) / 1e9, 3)
        if args.cells_rates:
            sweep = []
            for gbs in [float(x) for x in args.cells_rates.split(",")]:
                rate = gbs * 1e9
                row = {"rate_GBps": gbs}
                for name in ("layerwise", "chunkwise"):
                    if gbs * 1e9 == args.cap:
                        key = f"capped_{name}"
                        row[f"{name}_ms"] = round(ttft[key], 2)
                        continue
                    runs_r = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, 2, rate_bytes_per_s=rate,
                                      delivery=name, **kw)
                    row[f"{name}_ms"] = round(float(runs_r[1][1][0]["ttft_ms"]), 2)
                xr = [tp * b / rate * 1e3] * L
                row["eq3_ms"] = round(layerwise_floor(xr, c_ms), 2)
                row["chunkwise_model_ms"] = round(chunkwise_floor(xr, c_ms), 2)
                sweep.append(row)
            res["rate_sweep"] = sweep
            res["bandwidth_sensitivity"] = bandwidth_sensitivity(
                [{"rate_GBps": r["rate_GBps"], "layerwise_ms": [r["layerwise_ms"]],
                  "chunkwise_ms": [r["chunkwise_ms"]]} for r in sweep], 1.25, args.cap / 1e9)
        out["cells"].append(res)
        log(f"[bench] cell {ctx_len} @ {hit}: ttft {res['ttft_ms']} eq3 {res['eq3_ms']} "
            f"C/layer {res['compute_ms_per_layer']} ms X/layer {res['transfer_ms_per_layer_at_cap']} ms")
        del pool, table, q, kn, vn, outt, reqs, runs
        torch.cuda.empty_cache()
    return out


def cells_summary(path):
    """Markdown of a `--canonical-cells` JSON line (the file holds the
    script's stdout): per cell the four modes beside eq. (3) and the
    chunkwise form, then the layerwise/chunkwise rate sweep with the overlap
    requirement, then the 10-over-100 Gbps sensitivity."""
    with open(path) as f:
        d = json.loads([ln for ln in f.read().splitlines() if ln.startswith("{")][-1])["canonical_cells"]
    cap = d["cap_GBps"]
    out = [f"Llama-3-8B shape, random weights, G = {d['chunk_tokens']}, FFN {d['ffn_dim']}, cap {cap} GB/s.", "",
           "| C | hit | T_p / T_s | C_l (ms) | X_l (ms) | layer TFLOP/s | HBM | uncapped | capped LW | eq. (3) | "
           "capped CW | CW model | LW added over HBM |", "|" + "---|" * 13]
    name = {4096: "4K", 65536: "64K"}
    for c in d["cells"]:
        t = c["ttft_ms"]
        out.append(f"| {name.get(c['context'], c['context'])} | {c['hit'] * 100:g} % | {c['prefix_tokens']} / "
                   f"{c['suffix_tokens']} | {c['compute_ms_per_layer']} | {c['transfer_ms_per_layer_at_cap']} | "
                   f"{c['layer_tflops']} | {t['hbm_resident']} | {t['producer_uncapped']} | {t['capped_layerwise']} | "
                   f"{c['eq3_ms']} | {t['capped_chunkwise']} | {c['chunkwise_model_ms']} | "
                   f"{c['added_over_hbm_pct']['capped_layerwise']} % |")
    if any("rate_sweep" in c for c in d["cells"]):
        out += ["", "Rate sweep (ms; one timed trial per rate after a discarded first; B_req = layer bytes / C_l, "
                "the rate at which a layer's transfer equals its compute):", "",
                "| C | hit | B_req (GB/s) | rate (GB/s) | layerwise | eq. (3) | LW / eq. (3) | chunkwise | CW model |",
                "|" + "---|" * 9]
        for c in d["cells"]:
            for r in c.get("rate_sweep", []):
                out.append(f"| {name.get(c['context'], c['context'])} | {c['hit'] * 100:g} % | {c['required_GBps']} | "
                           f"{r['rate_GBps']} | {r['layerwise_ms']} | {r['eq3_ms']} | "
                           f"{r['layerwise_ms'] / r['eq3_ms']:.3f} | {r['chunkwise_ms']} | {r['chunkwise_model_ms']} |")
        out += ["", "Bandwidth sensitivity: TTFT at 1.25 GB/s (10 Gbps) over 12.5 GB/s (100 Gbps), minus one:", "",
                "| C | hit | B_req (GB/s) | layerwise | chunkwise |", "|---|---|---|---|---|"]
        for c in d["cells"]:
            sens = c.get("bandwidth_sensitivity")
            if sens:
                out.append(f"| {name.get(c['context'], c['context'])} | {c['hit'] * 100:g} % | {c['required_GBps']} | "
                           f"+{sens['layerwise_increase'] * 100:.1f} % | +{sens['chunkwise_increase'] * 100:.1f} % |")
    return "\n".join(out)


def cpu_model():
    """The host CPU as lscpu reports it: the model name, then the family,
    model and stepping numbers and the CPU count (a virtual machine may show
    only a generic model name); else /proc/cpuinfo's model name."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        f = {}
        for ln in out.splitlines():
            if ":" in ln:
                k, v = ln.split(":", 1)
                f.setdefault(k.strip(), v.strip())
        if f.get("Model name"):
            ids = ", ".join(f"{k.lower()} {f[k]}" for k in ("CPU family", "Model", "Stepping") if f.get(k))
            extra = "; ".join(x for x in (ids, f"{f['CPU(s)']} CPUs" if f.get("CPU(s)") else "") if x)
            return f"{f['Model name']} ({extra})" if extra else f["Model name"]
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as fh:
            return next((ln.split(":", 1)[1].strip() for ln in fh if ln.startswith("model name")), "unknown")
    except OSError:
        return "unknown"


def cpu_baseline(wl, objs_all, tables, budget_s):
    """The CPU oracle, as it stands, on a bounded sample of the same workload."""
    import oracle
    L, nq, nkv, d, G, Ps = (wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.chunk_tokens,
                            wl.page_size)
    objs, table = objs_all[0], tables[0]
    n = objs.shape[0]
    tp = wl.prefix_tokens[0]
    pool = np.zeros(oracle.pool_shape(1, wl.pool_pages, nkv, Ps, d), dtype=np.uint16)
    threads = min(16, len(os.sched_getaffinity(0)))     # the host share of one GPU
    layers, secs = 0, 0.0
    while layers < L and (layers == 0 or secs < budget_s * 0.5):
        staging = np.ascontiguousarray(objs[:, layers, :]).reshape(-1)
        t = time.perf_counter()
        oracle.ingest_layer(staging, n, G, nkv, d, Ps, table, pool, 0, threads=threads)
        secs += time.perf_counter() - t
        layers += 1
    ingest_gbs = 2.0 * layers * tp * 2 * nkv * d * 2 / secs / 1e9
    # attention: a few suffix rows of layer 0 over the whole prefix, all heads
    import kvgen
    ts = wl.suffix_tokens[0]
    q = kvgen.suffix_tensor(wl.seed, kvgen.KIND_Q, 0, 0, (ts, nq, d))
    kn = kvgen.suffix_tensor(wl.seed, kvgen.KIND_KNEW, 0, 0, (ts, nkv, d))
    vn = kvgen.suffix_tensor(wl.seed, kvgen.KIND_VNEW, 0, 0, (ts, nkv, d))
    chunks = [np.ascontiguousarray(objs[j]).reshape(-1) for j in range(n)]
    k, v = oracle.logical_kv(chunks, G, nkv, d, 0)
    rows, flops, asecs = [], 0.0, 0.0
    step = max(1, ts // 64)
    for i in range(ts - 1, -1, -step):
        if asecs > budget_s * 0.5 and rows:
            break
        t = time.perf_counter()
        oracle.attention(q, k, v, kn, vn, rows=[i], threads=threads)
        asecs += time.perf_counter() - t
        rows.append(i)
        flops += 4.0 * nq * d * (tp + i + 1)
    cpu = cpu_model()
    rate = flops / asecs                                    # flop/s of the sampled rows
    layer_flops = attn_flops(nq, d, tp, ts)
    return {
        "value": round(ingest_gbs, 4), "unit": "GB/s", "cores": threads, "kind": "oracle", "cpu": cpu,
        "sample": f"oracle byte-loop ingest ({threads} threads over the chunks) of {layers} of {L} layer "
                  f"payloads of request 0 ({layers * tp} tokens x {2 * nkv * d * 2} B, read + written)",
        "attention": {"gflops": round(rate / 1e9, 4), "cores": threads, "rows": len(rows),
                      "sample": f"float64 attention of {len(rows)} suffix rows x {nq} heads of layer 0 over "
                                f"{tp} prefix keys, {threads} threads",
                      "layer_s_extrapolated": round(layer_flops / rate, 2),
                      "all_layers_s_extrapolated": round(L * layer_flops / rate, 1)},
        "seconds": round(secs + asecs, 2),
    }


def attention_rate(wl, runs):
    """TFLOP/s and ms of one layer's attention over HBM-resident runs: from
    the first event before a layer's attention to the last one after it (one
    launch when requests are batched, one after another otherwise)."""
    L, R = wl.num_layers, wl.n_requests
    op_ms, op_flops = 0.0, 0.0
    for _, st in runs:
        for l in range(L):
            op_ms += max(rst["done_ms"][l] for rst in st) - min(rst["ingested_ms"][l] for rst in st)
            op_flops += sum(attn_flops(wl.num_q_heads, wl.head_dim, wl.prefix_tokens[r], wl.suffix_tokens[r])
                            for r in range(R))
    return op_flops / (op_ms / 1e3) / 1e12, op_ms / (len(runs) * L)


def zero_kv(args):
    """HBM-resident runs over an all-zero pool, then over the same pool after
    the device-staged pipeline has ingested the N(0,1) payloads.  The kernels
    and their launch shapes are the same; only the K/V values differ."""
    import kvgen
    import paper_2605_22850_amd as oc
    wl = kvgen.workload(args.workload)
    layout, pool, reqs, _, _ = setup(wl)
    trials = max(2, args.trials)
    out = {}
    for name in ("zero", "ingested"):
        if name == "ingested":
            run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_DEVICE_STAGED, 1)
        runs = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_HBM_RESIDENT, trials)[1:]
        tflops, ms = attention_rate(wl, runs)
        out[name] = {"ttft_ms": mean_std([r[0] for r in runs]), "attention_tflops": round(tflops, 2),
                     "attention_ms_per_layer": round(ms, 4)}
        log(f"[bench] {name} pool: {out[name]}")
    return {"workload": wl.name, "trials": trials - 1, **out}


def ingest_tables(args):
    """The isolated ingest of the main workload with its own (seeded random)
    block table and with the identity table (prefix page j in pool page j),
    same payloads and launch shape, beside a plain device copy of the same
    bytes: what the table's page placement costs the kernel.  `--tables`
    picks the tables (one per counter run)."""
    import torch
    import kvgen
    import paper_2605_22850_amd as oc
    torch.cuda.set_device(0)
    wl = kvgen.workload(args.workload)
    layout, pool, reqs, _, _ = setup(wl)
    L, b = wl.num_layers, 2 * wl.num_kv_heads * wl.head_dim * 2
    out = {"workload": wl.name, "tables": {}}
    for name in args.tables.split(","):
        if name == "identity":
            for rq in reqs:
                rq.pages = torch.arange(rq.pages.numel(), dtype=torch.int32, device="cuda")
        elif name != "random":
            raise SystemExit(f"unknown table {name}")
        out["tables"][name] = isolated_ingest(oc, wl, layout, pool, reqs, args.isolated_passes)
        log(f"[bench] ingest with the {name} table: {out['tables'][name]['value']} GB/s")
    # plain copy of the same bytes per launch (payload layer -> a buffer), layers rotated
    s = torch.cuda.Stream()
    tp = wl.prefix_tokens[0]
    dst = torch.empty(tp * b // 2, dtype=torch.int16, device="cuda")
    launches = [(lambda l=l: dst.copy_(reqs[0].device_payload[l * tp * b // 2:(l + 1) * tp * b // 2]),
                 2.0 * tp * b) for l in range(L)]
    with torch.cuda.stream(s):
        warm_device(s, lambda: [fn() for fn, _ in launches])
        evs, _ = gated_passes(s, launches, args.isolated_passes)
    out["plain_copy"] = _rate(evs, "device-to-device copy of each layer payload (torch copy_), same bytes")
    return out


def ingest_tables_summary(paths):
    """Markdown of rocprofv3 counter databases of `--ingest-tables` runs, one
    table per run: mean per ingest dispatch of every counter collected."""
    import sqlite3
    out = ["| run | dispatches | mean us | counter | mean per dispatch |", "|---|---|---|---|---|"]
    for path in paths:
        c = sqlite3.connect(path)
        rows = list(c.execute("select dispatch_id,kernel_name,counter_name,value,start,end "
                              "from counters_collection order by start"))
        by_disp = {}
        for disp, name, cn, val, st, en in rows:
            if "kv_ingest" not in name:
                continue
            e = by_disp.setdefault(disp, {"dur": en - st, "c": {}})
            e["c"][cn] = e["c"].get(cn, 0.0) + val
        disp = list(by_disp.values())
        label = os.path.basename(os.path.dirname(path)) or os.path.basename(path)
        dur = np.mean([e["dur"] for e in disp]) / 1e3 if disp else float("nan")
        for cn in sorted({k for e in disp for k in e["c"]}):
            out.append(f"| {label} | {len(disp)} | {dur:.1f} | {cn} | "
                       f"{np.mean([e['c'][cn] for e in disp if cn in e['c']]):.4g} |")
        # average latencies (cycles) where a pass holds both the summed
        # in-flight level (or latency) and the request count (Little's law)
        for what, lev, cnt in LATENCY_PAIRS:
            pairs = [e["c"][lev] / e["c"][cnt] for e in disp if e["c"].get(cnt, 0) > 0 and lev in e["c"]]
            if pairs:
                out.append(f"| {label} | {len(disp)} | {dur:.1f} | {what} (= {lev} / {cnt}) | {np.mean(pairs):.4g} |")
    return "\n".join(out)


LATENCY_PAIRS = [
    ("memory-side read latency", "TCC_EA0_RDREQ_LEVEL_sum", "TCC_EA0_RDREQ_sum"),
    ("memory-side write latency", "TCC_EA0_WRREQ_LEVEL_sum", "TCC_EA0_WRREQ_sum"),
    ("L1 -> L2 read latency", "TCP_TCC_READ_REQ_LATENCY_sum", "TCP_TCC_READ_REQ_sum"),
    ("L1 -> L2 write latency", "TCP_TCC_WRITE_REQ_LATENCY_sum", "TCP_TCC_WRITE_REQ_sum"),
]


def step_ingest(stats_all, wl):
    """In-step ingest of timed pipeline runs: algorithmic bytes (read + write
    of every layer payload) over the summed time between each layer's landed
    and ingested events on the copy stream.  Requests whose layer is ingested
    by one launch together report the same pair of events; it counts once."""
    L, b = wl.num_layers, 2 * wl.num_kv_heads * wl.head_dim * 2
    ingest_ms, n = 0.0, 0
    for st in stats_all:
        for l in range(L):
            for t0, t1 in sorted({(rst["landed_ms"][l], rst["ingested_ms"][l]) for rst in st}):
                ingest_ms += t1 - t0
                n += 1
    nbytes = 2.0 * sum(wl.prefix_tokens) * b * L * len(stats_all)
    gbs = nbytes / (ingest_ms / 1e3) / 1e9
    return {"value": round(gbs, 2), "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "launches": n,
            "mean_launch_us": round(ingest_ms / n * 1e3, 3), "bytes_per_launch": nbytes / n}


def workload_legs(oc, name, args):
    """One more workload, every figure the main one reports: timed
    device-staged steps (in-step ingest), the four TTFT modes with the gates,
    the attention rate and the isolated ingest.  Frees its device memory."""
    import torch
    import kvgen
    wl = kvgen.workload(name)
    L, nq, d, R = wl.num_layers, wl.num_q_heads, wl.head_dim, wl.n_requests
    layout, pool, reqs, _, _ = setup(wl)
    buf = torch.empty(1 << 27, dtype=torch.int16, device="cuda")
    warm_device(torch.cuda.current_stream(), lambda: buf.fill_(1))
    del buf
    run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_DEVICE_STAGED, 2)
    ctx = oc.oc_context_create(pool, layout, oc.OC_MODE_DEVICE_STAGED, max(wl.prefix_tokens),
                               max(wl.suffix_tokens), **RUN_OPTS)
    steps = max(2, args.other_steps)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    stats_all = [oc.oc_pipeline_run(ctx, reqs, L) for _ in range(steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    oc.oc_context_destroy(ctx)
    out = {"workload": wl.name, "layers": L, "q_heads": nq, "kv_heads": wl.num_kv_heads, "head_dim": d,
           "prefix_tokens": wl.prefix_tokens if R > 1 else wl.prefix_tokens[0],
           "suffix_tokens": wl.suffix_tokens if R > 1 else wl.suffix_tokens[0],
           "steps": steps, "ms_per_step": round(wall / steps * 1e3, 3),
           "ingest_in_step": step_ingest(stats_all, wl)}
    trials = max(2, args.trials)
    hbm = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_HBM_RESIDENT, trials)
    dev = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_DEVICE_STAGED, trials)
    tflops, op_ms = attention_rate(wl, hbm[1:])
    out["attention"] = {"roofline": {"bound": "mfma", "achieved": round(tflops, 2), "peak": BF16_PEAK_TFLOPS,
                                     "unit": "TFLOP/s", "frac": round(tflops / BF16_PEAK_TFLOPS, 4)},
                        "op_ms_per_layer": round(op_ms, 4),
                        "launch": "one per layer for all requests" if R > 1 and not RUN_OPTS.get(
                            "attention_per_request") else "one per request and layer"}
    out["ttft_ms"], res = ttft_legs(oc, wl, layout, pool, reqs, args, hbm, dev, sweep=False)
    out.update(res)
    if args.isolated_passes > 0:
        out["ingest_isolated"] = isolated_ingest(oc, wl, layout, pool, reqs, max(2, args.isolated_passes))
    del pool, reqs, hbm, dev
    torch.cuda.empty_cache()
    log(f"[bench] {wl.name} legs done")
    return out


def run_bench(args):
    import torch
    import kvgen
    import paper_2605_22850_amd as oc

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    wl = kvgen.workload(args.workload)
    L, nq, nkv, d, R = wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.n_requests
    b = 2 * nkv * d * 2
    layout, pool, reqs, objs_all, tables = setup(wl)
    if args.copy_calibration:
        copy_calibration()
        log("[bench] copy calibration done")

    # ---- timed steps: device-staged pipeline, all layers ----
    # the device leaves its idle clocks first (host-side setup kept it idle
    # for seconds): WARM_S of plain fills (no ingest or copy launch, so the
    # profile summaries still find the timed steps and the calibration copies
    # by launch order), then the warmup steps
    buf = torch.empty(1 << 27, dtype=torch.int16, device="cuda")
    warm_device(torch.cuda.current_stream(), lambda: buf.fill_(1))
    del buf
    for i in range(args.warmup):
        run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_DEVICE_STAGED, 1)
        log(f"[bench] warmup {i + 1}/{args.warmup}")
    ctx = oc.oc_context_create(pool, layout, oc.OC_MODE_DEVICE_STAGED, max(wl.prefix_tokens),
                               max(wl.suffix_tokens), **RUN_OPTS)
    stats_all = []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        stats_all.append(oc.oc_pipeline_run(ctx, reqs, L))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    oc.oc_context_destroy(ctx)
    log(f"[bench] {args.steps} steps in {wall:.3f} s")
    ingest_ms, n_ingest = 0.0, 0
    for st in stats_all:
        for rst in st:
            for l in range(L):
                ingest_ms += rst["ingested_ms"][l] - rst["landed_ms"][l]
                n_ingest += 1
    ingest_bytes_per_step = 2.0 * sum(wl.prefix_tokens) * b * L       # read + write, every layer
    value = ingest_bytes_per_step * args.steps / (ingest_ms / 1e3) / 1e9
    per_launch_bytes = ingest_bytes_per_step / (L * R)
    mean_launch_us = ingest_ms / n_ingest * 1e3
    traffic, traffic_src = read_traffic(wl.name)
    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(wall / args.steps * 1e3, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded N(0,1) bf16 KV/Q, Fisher-Yates block tables",
        "config": {"workload": wl.name, "layers": L, "q_heads": nq, "kv_heads": nkv, "head_dim": d,
                   "prefix_tokens": wl.prefix_tokens if R > 1 else wl.prefix_tokens[0],
                   "suffix_tokens": wl.suffix_tokens if R > 1 else wl.suffix_tokens[0],
                   "page_tokens": wl.page_size, "chunk_tokens": wl.chunk_tokens, "pool_pages": wl.pool_pages,
                   "step": "device-staged pipeline: per layer ingest (copy stream) then attention (compute "
                           "stream), all layers"},
        "roofline": {"bound": "hbm", "kernel": "ingest (kv_ingest_rows_kernel beside the attention; "
                     "kv_ingest_src_kernel for a step's first layer)", "achieved": round(value, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(value / HBM_PEAK_GBS, 4),
                     "traffic": traffic, "traffic_source": traffic_src,
                     "bytes_per_launch": per_launch_bytes, "launches": n_ingest,
                     "mean_launch_us": round(mean_launch_us, 3)},
    }

    # ---- TTFT modes ----
    trials = max(2, args.trials)
    hbm = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_HBM_RESIDENT, trials)
    log("[bench] hbm-resident trials done")
    dev = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_DEVICE_STAGED, trials)
    log("[bench] device-staged trials done")
    t_hbm = [x[0] for x in hbm[1:]]
    t_dev = [x[0] for x in dev[1:]]
    # attention of a layer, all requests: from the first event before it to
    # the last one after it (one launch when requests are batched, one after
    # another otherwise), HBM-resident
    attn_tflops, op_ms_layer = attention_rate(wl, hbm[1:])
    flops_per_layer = sum(attn_flops(nq, d, wl.prefix_tokens[r], wl.suffix_tokens[r]) for r in range(R))
    layer_tflops = flops_per_layer / (sum(t_hbm) / len(t_hbm) / L / 1e3) / 1e12
    line["attention"] = {
        "roofline": {"bound": "mfma", "achieved": round(attn_tflops, 2), "peak": BF16_PEAK_TFLOPS,
                     "unit": "TFLOP/s", "frac": round(attn_tflops / BF16_PEAK_TFLOPS, 4)},
        "flops_per_layer": flops_per_layer, "op_ms_per_layer": round(op_ms_layer, 4),
        "what": "attention + split combine of one layer (all requests), HIP events around them",
        "tflops_whole_pass": round(layer_tflops, 2),
    }
    line["ttft_ms"], res = ttft_legs(oc, wl, layout, pool, reqs, args, hbm, dev)
    line.update(res)
    if args.policy_sweep:
        line["policy_sweep"] = policy_sweep(oc, wl, layout, pool, reqs, args, hbm)
    del hbm, dev
    if args.isolated_passes > 0:
        line["ingest_isolated"] = isolated_ingest(oc, wl, layout, pool, reqs, args.isolated_passes)
        log("[bench] isolated ingest done")
        if wl.name != "tiny":
            # 128 KiB per layer: L2-resident and bound by launch latency
            wl3 = kvgen.workload("tiny")
            lay3, pool3, reqs3, _, _ = setup(wl3)
            line["tiny_ingest_isolated"] = isolated_ingest(oc, wl3, lay3, pool3, reqs3, 50)
            del pool3, reqs3
        line["write_path"] = write_path(oc, wl, layout, pool, reqs, args.isolated_passes)
        log("[bench] write path done")
    # the other workloads, one at a time (the main one's device memory freed first)
    others = [w for w in args.other_workloads.split(",") if w and w != wl.name]
    if others:
        del pool, reqs
        torch.cuda.empty_cache()
        line["workloads"] = {w: workload_legs(oc, w, args) for w in others}
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle) ...")
        line["cpu_baseline"] = cpu_baseline(wl, objs_all, tables, args.cpu_budget)
    print(json.dumps(line), flush=True)


# ---------------------------------------------------------------------------
# rocprofv3 output -> markdown
# ---------------------------------------------------------------------------

def _short(name):
    n = name.replace("void ", "")
    if n.startswith("at::native"):
        return "torch " + ("fill" if "Fill" in n else "elementwise")
    return n.split("(")[0]


def marker_summary(paths):
    """Markdown summary of a rocprofv3 --marker-trace --kernel-trace
    (--memory-copy-trace) database: the library's roctx ranges (each pipeline
    run, each layer's wait and enqueue) and marks (each payload the producer
    completes), set against the kernels and host-to-device copies.  Per run:
    the host time of the run and of its layer ranges; with a producer, the gap
    between payload marks (the delivery interval), the DMA spans of each layer
    and the lag from a payload's mark to its last span landing and to its
    ingest launch (one request delivered in layer order)."""
    import sqlite3

    def message(extdata):
        try:
            return json.loads(extdata or "{}").get("message", "")
        except ValueError:
            return ""

    out = []
    for path in paths:
        c = sqlite3.connect(path)
        # ranges are regions, marks are samples; the roctx message is in extdata
        regs = [(message(x), tid, st, en) for x, tid, st, en in
                c.execute("select extdata,tid,start,end from regions order by start")]
        marks = [(message(x), tid, ts) for x, tid, ts in
                 c.execute("select extdata,tid,timestamp from samples order by timestamp")]
        kern = list(c.execute("select name,start,end from kernels order by start"))
        # host-to-device copies, when the trace has them (--memory-copy-trace)
        copies = [(st, en, size) for st, en, size, kind in
                  c.execute("select start,end,size,src_agent_type from memory_copies order by start")
                  if kind == "CPU"]
        out.append(f"### Markers: `{os.path.basename(path)}`\n")
        kinds = {}
        for msg, *_ in regs:
            key = ("range", msg.split(" ")[0])
            kinds[key] = kinds.get(key, 0) + 1
        for msg, *_ in marks:
            key = ("mark", msg.split(" ")[0])
            kinds[key] = kinds.get(key, 0) + 1
        out.append("| roctx | message starts | count |\n|---|---|---|")
        for (kind, head), n in sorted(kinds.items()):
            out.append(f"| {kind} | `{head}` | {n} |")
        out.append("")
        runs = [r for r in regs if r[0] == "oc_pipeline_run"]
        out.append("| run | host ms | layer ranges | mean layer range us | payload marks | mean mark gap ms | "
                   "DMA spans per layer | DMA GB/s | mark -> last span landed us | last span -> ingest start us | "
                   "mark -> ingest start us (max) |\n|---|---|---|---|---|---|---|---|---|---|---|")
        for i, (_, tid, st, en) in enumerate(runs):
            lay = [r for r in regs if st <= r[2] <= en and r[1] == tid and r[0].startswith("layer ")]
            ts = [m[2] for m in marks if st <= m[2] <= en and m[0].startswith("ready ")]
            cps = [x for x in copies if st <= x[0] <= en]
            ing = [k[1] for k in kern if st <= k[1] <= en and "kv_ingest" in k[0]]
            row = f"| {i} | {(en - st) / 1e6:.2f} | {len(lay)} | "
            row += f"{np.mean([r[3] - r[2] for r in lay]) / 1e3:.1f} | " if lay else "- | "
            row += f"{len(ts)} | "
            row += f"{np.mean(np.diff(ts)) / 1e6:.3f} | " if len(ts) >= 2 else "- | "
            # one request delivered in layer order: the i-th payload mark and
            # the i-th ingest launch are one layer's, and the copy stream runs
            # that layer's DMA spans between the previous ingest and its own
            if ts and cps and len(ts) == len(ing):
                spans, land, to_ing, lag, prev = [], [], [], [], -1
                for m, k0 in zip(ts, ing):
                    mine = [x for x in cps if prev < x[1] <= k0]
                    prev = k0
                    if not mine:
                        continue
                    spans.append(len(mine))
                    land.append(mine[-1][1] - m)
                    to_ing.append(k0 - mine[-1][1])
                    lag.append(k0 - m)
                nb = float(sum(x[2] for x in cps))
                dma = float(sum(x[1] - x[0] for x in cps))
            if ts and cps and len(ts) == len(ing) and spans:
                row += (f"{np.mean(spans):.1f} | {nb / dma:.1f} | {np.mean(land) / 1e3:.1f} | "
                        f"{np.mean(to_ing) / 1e3:.1f} | {np.mean(lag) / 1e3:.1f} ({np.max(lag) / 1e3:.1f}) |")
            else:
                row += "- | - | - | - | - |"
            out.append(row)
        out.append("")
    return "\n".join(out)


def profile_summary(paths, workload, warmup, steps):
    import sqlite3
    import kvgen
    wl = kvgen.workload(workload)
    per_run = wl.num_layers * sum(1 for t in wl.prefix_tokens if t > 0)
    lo, hi = warmup * per_run, (warmup + steps) * per_run
    b = 2 * wl.num_kv_heads * wl.head_dim * 2
    out = []
    counters = {}
    attn_counters = []
    clock_runs = []
    for path in paths:
        c = sqlite3.connect(path)
        has_pmc = c.execute("select count(*) from counters_collection").fetchone()[0] > 0
        if not has_pmc:
            out.append(f"### Kernel trace: `{os.path.basename(path)}`\n")
            out.append("| kernel | calls | total ms | average us | % |\n|---|---|---|---|---|")
            for name, calls, tot, avg, pct in c.execute(
                    "select name,total_calls,total_duration,average,percentage from top_kernels"):
                # this view reports microseconds
                out.append(f"| `{_short(name)}` | {calls} | {tot / 1e3:.3f} | {avg:.3f} | {pct:.2f} |")
            rows = list(c.execute("select name,start,end,vgpr_count,accum_vgpr_count,lds_size,grid_x "
                                  "from kernels order by start"))
            # both ingest launch shapes (alone / beside the attention) count as the ingest
            ing = [r for r in rows if "kv_ingest" in r[0]]
            att = [r for r in rows if "attn_fwd_kernel" in r[0]]
            out.append("")
            for label, ks in (("ingest", ing), ("attn_fwd_kernel", att)):
                sel = ks[lo:hi]
                if not sel:
                    continue
                dur = [(r[2] - r[1]) / 1e3 for r in sel]
                out.append(f"- {label} in the timed steps (launches {lo}..{hi - 1} in start order, "
                           f"warmup {warmup} x {per_run} skipped): {len(sel)} launches, mean {np.mean(dur):.3f} us, "
                           f"min {min(dur):.3f}, max {max(dur):.3f}")
                for name in sorted({_short(r[0]) for r in sel}):
                    part = [r for r in sel if _short(r[0]) == name]
                    d2 = [(r[2] - r[1]) / 1e3 for r in part]
                    out.append(f"  - `{name}`: {len(part)} launches, mean {np.mean(d2):.3f} us; VGPR {part[0][3]}, "
                               f"AGPR {part[0][4]}, LDS {part[0][5]} B, grid {part[0][6]} threads")
                if label == "ingest":
                    nbytes = 2.0 * sum(wl.prefix_tokens) * b / len(wl.prefix_tokens)
                    out.append(f"  - algorithmic bytes per launch {nbytes:.0f} -> "
                               f"{nbytes / (np.mean(dur) * 1e-6) / 1e9:.1f} GB/s over the timed launches")
            out.append("")
        else:
            rows = list(c.execute("select dispatch_id,kernel_name,counter_name,value,start,end "
                                  "from counters_collection order by start"))
            by_disp = {}
            for disp, name, cn, val, st, en in rows:
                e = by_disp.setdefault(disp, {"name": name, "start": st, "end": en, "c": {}})
                e["c"][cn] = e["c"].get(cn, 0.0) + val
            disp = sorted(by_disp.values(), key=lambda e: e["start"])
            if any("GRBM_GUI_ACTIVE" in e["c"] for e in disp):
                clock_runs.append((os.path.basename(path), disp))
            att = [e for e in disp if "attn_fwd_kernel" in e["name"]][lo:hi]
            if att and any(e["c"] for e in att):
                attn_counters.append((os.path.basename(path), att))
            ing = [e for e in disp if "kv_ingest" in e["name"]]
            first_ing = ing[0]["start"] if ing else float("inf")
            cal = [e for e in disp if "copyBuffer" in e["name"] and e["start"] < first_ing
                   and e["end"] - e["start"] > 20000]
            sel = ing[lo:hi]
            for cn in sorted({k for e in sel for k in e["c"]} & {"FETCH_SIZE", "WRITE_SIZE"}):
                counters[cn] = {"ingest_kib": float(np.mean([e["c"][cn] for e in sel])),
                                "calib_kib": float(sum(e["c"].get(cn, 0.0) for e in cal)),
                                "calib_dispatches": len(cal), "ingest_dispatches": len(sel),
                                "db": os.path.basename(path)}
    for db, att in attn_counters:
        # derived counters as rocprofv3 reports them (percent of the kernel's GPU time)
        flops = attn_flops(wl.num_q_heads, wl.head_dim, wl.prefix_tokens[0], wl.suffix_tokens[0])
        out.append(f"### Attention counters (`{db}`, {len(att)} timed-step `attn_fwd_kernel` dispatches)\n")
        out.append("| counter | mean per dispatch |\n|---|---|")
        for cn in sorted({k for e in att for k in e["c"]}):
            vals = [e["c"][cn] for e in att if cn in e["c"]]
            out.append(f"| {cn} | {np.mean(vals):.4g} |")
        dur_ns = float(np.mean([e["end"] - e["start"] for e in att]))
        out.append(f"| (mean dispatch duration, ns) | {dur_ns:.4g} |")
        mops = [e["c"]["SQ_INSTS_VALU_MFMA_MOPS_BF16"] for e in att if "SQ_INSTS_VALU_MFMA_MOPS_BF16" in e["c"]]
        if mops:
            out.append("")
            out.append(f"MFMA bf16 flops per dispatch (MOPS x 512): {np.mean(mops) * 512:.4g}; algorithmic "
                       f"flops per layer (unmasked pairs): {flops:.4g}; ratio {np.mean(mops) * 512 / flops:.3f} "
                       f"(masked pairs of the causal diagonal and padding rows are computed and discarded).")
        out.append("")
    for db, disp in clock_runs:
        # GPU clock cycles counted while a dispatch ran, per nanosecond of its
        # duration: proportional to the clock the chip ran that kernel at
        out.append(f"### Clock counter by run (`{db}`; launches grouped {per_run} per pipeline run, "
                   f"in start order)\n")
        out.append("| kernel | run | launches | mean us | GRBM_GUI_ACTIVE per ns |\n|---|---|---|---|---|")
        for label in ("attn_fwd_kernel", "kv_ingest"):
            ks = [e for e in disp if label in e["name"] and "GRBM_GUI_ACTIVE" in e["c"]]
            for i in range(0, len(ks), per_run):
                part = ks[i:i + per_run]
                dur = np.array([e["end"] - e["start"] for e in part], dtype=float)
                act = np.array([e["c"]["GRBM_GUI_ACTIVE"] for e in part])
                out.append(f"| `{label}` | {i // per_run} | {len(part)} | {dur.mean() / 1e3:.1f} | "
                           f"{np.mean(act / dur):.3f} |")
        out.append("")
    if counters:
        nbytes = 2.0 * sum(wl.prefix_tokens) * b / len(wl.prefix_tokens)
        out.append("### HBM byte counters (ingest, timed-step launches)\n")
        out.append("| counter | per ingest launch (KiB) | calibration copies (KiB) | scale | "
                   "scaled bytes per launch |\n|---|---|---|---|---|")
        total = 0.0
        for cn, v in counters.items():
            expect = CALIB_COPIES * CALIB_BYTES / 1024.0
            scale = expect / v["calib_kib"] if v["calib_kib"] > 0 else float("nan")
            scaled = v["ingest_kib"] * 1024.0 * scale
            total += scaled
            out.append(f"| {cn} | {v['ingest_kib']:.0f} | {v['calib_kib']:.0f} ({v['calib_dispatches']} "
                       f"dispatches) | {scale:.4f} | {scaled:.0f} |")
        out.append("")
        out.append(f"Algorithmic bytes per launch: {nbytes:.0f} (read + write of the layer payload); "
                   f"measured / algorithmic = {total / nbytes:.4f}.\n")
        if len(counters) >= 2:
            out.append(f"traffic_bytes_per_launch: {total:.0f}")
            out.append(f"kernel_source_sha256: {file_sha256(INGEST_SRC)}")
    return "\n".join(out)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="8b-64k")
    ap.add_argument("--trials", type=int, default=6, help="TTFT trials per mode; the first is excluded")
    ap.add_argument("--cap", type=float, default=12.5e9, help="producer rate cap, bytes/s (12.5e9 = 100 Gbps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-producer", action="store_true", help="skip the producer TTFT modes")
    ap.add_argument("--isolated-passes", type=int, default=2, help="passes of the isolated ingest leg (0: skip)")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--sweep-rates", default="1.25,12.5,50,0",
                    help="producer rates (GB/s, 0 = uncapped) of the layerwise/chunkwise sweep; empty: skip")
    ap.add_argument("--sweep-max-s", type=float, default=8.0, help="skip sweep rates whose payload takes longer")
    ap.add_argument("--policy-sweep", action="store_true",
                    help="run every bandwidth allocation policy under the cap (meant for --workload batch8)")
    ap.add_argument("--scheduler-workloads", default="",
                    help="run the multi-tenant scheduler evaluation on these workloads (e.g. A,B,C) instead")
    ap.add_argument("--scheduler-scale", type=int, default=4,
                    help="divide the scheduler workloads' cached tokens and compute windows by this")
    ap.add_argument("--canonical-cells", action="store_true",
                    help="run the end-to-end TTFT cells (4K/64K x 12.5/50/87.5%% hits) with the whole layer's "
                         "compute instead")
    ap.add_argument("--cells-chunk", type=int, default=64, help="chunk tokens G of the canonical cells")
    ap.add_argument("--cells-rates", default="1.25,2.5,5,12.5,25,50",
                    help="producer rates (GB/s) of the canonical cells' layerwise/chunkwise sweep ('' to skip); "
                         "one timed trial each after a discarded first")
    ap.add_argument("--policy-margin", type=float, default=0.625e9,
                    help="Calibrated Stall-opt margin, bytes/s (0.625e9 = 5 Gbps)")
    ap.add_argument("--other-workloads", "--second-workload", dest="other_workloads",
                    default="8b-4k,batch8,70b-32k",
                    help="workloads whose steps, TTFT legs, attention and isolated ingest are reported beside "
                         "the main one, comma-separated ('' to skip)")
    ap.add_argument("--other-steps", type=int, default=5, help="timed device-staged steps of each other workload")
    ap.add_argument("--copy-calibration", action="store_true",
                    help=f"{CALIB_COPIES} plain {CALIB_BYTES >> 20} MiB device copies before the steps")
    ap.add_argument("--attention-per-request", action="store_true",
                    help="one attention launch per request and layer, not one per layer for all requests")
    ap.add_argument("--zero-kv", action="store_true",
                    help="HBM-resident runs over an all-zero pool, then over the ingested N(0,1) pool")
    ap.add_argument("--tables", default="",
                    help="isolated ingest of the workload with these block tables instead (random,identity)")
    ap.add_argument("--ingest-tables-summary", nargs="+", metavar="DB",
                    help="print a markdown summary of rocprofv3 counter databases of --tables runs")
    ap.add_argument("--cells-summary", metavar="JSON",
                    help="print a markdown summary of a saved --canonical-cells output line (no GPU needed)")
    ap.add_argument("--marker-summary", nargs="+", metavar="DB",
                    help="print a markdown summary of the roctx ranges and marks in rocprofv3 databases")
    ap.add_argument("--profile-summary", nargs="+", metavar="DB",
                    help="print a markdown summary of rocprofv3 databases of a run of this script")
    args = ap.parse_args()

    if args.marker_summary:
        print(marker_summary(args.marker_summary))
        return
    if args.profile_summary:
        print(profile_summary(args.profile_summary, args.workload, args.warmup, args.steps))
        return
    if args.cells_summary:
        print(cells_summary(args.cells_summary))
        return
    if args.ingest_tables_summary:
        print(ingest_tables_summary(args.ingest_tables_summary))
        return
    if args.attention_per_request:
        RUN_OPTS["attention_per_request"] = True
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the path has no cross-GPU part; run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)
    if args.canonical_cells:
        res = canonical_cells(args)
        print(json.dumps({"metric": "TTFT with the whole layer's compute, end-to-end cells", "unit": "ms",
                          "higher_is_better": False, "data": "synthetic: random weights and KV", "n_gpus": 1,
                          "canonical_cells": res}), flush=True)
        return
    if args.tables:
        print(json.dumps({"metric": "isolated ingest by block table", "unit": "GB/s", "higher_is_better": True,
                          "data": "synthetic", "n_gpus": 1, "ingest_tables": ingest_tables(args)}), flush=True)
        return
    if args.zero_kv:
        print(json.dumps({"metric": "attention per layer over zero vs N(0,1) K/V", "unit": "TFLOP/s",
                          "higher_is_better": True, "data": "synthetic", "n_gpus": 1,
                          "zero_kv": zero_kv(args)}), flush=True)
        return
    if args.scheduler_workloads:
        res = scheduler_workloads(args)
        print(json.dumps({"metric": "added TTFT by bandwidth allocation policy (scheduler workloads)",
                          "unit": "ms", "higher_is_better": False, "data": "synthetic", "n_gpus": 1,
                          "scheduler_workloads": res}), flush=True)
        return
    run_bench(args)


if __name__ == "__main__":
    main()
