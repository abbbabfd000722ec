#!/usr/bin/env python3
"""Benchmark of the layerwise prefix-KV hot path on one MI355X.

A step is one pass of the whole path over one request with its payloads
already in HBM: for every layer, ingest (unpack + scatter into the paged
pool) on the copy stream, then that layer's suffix-prefill attention on the
compute stream as soon as the layer's ingested event fires -- all layers,
two streams, per-layer events.

Reported (one JSON line):
  value            KV ingest GB/s = algorithmic bytes (read + write of every
                   layer payload) / summed ingest kernel time, timed with HIP
                   events on the copy stream over the timed steps
  roofline         ingest against 8 TB/s HBM
  attention        attention TFLOP/s (attention-only pass) against 2.5 PFLOP/s
  ttft_ms          HBM-resident / device-staged / producer uncapped / producer
                   capped at 12.5 GB/s (100 Gbps), mean and std over trials
                   after the first
  added_ttft_ms    capped producer minus HBM-resident, and the eq. (3) floor
  cpu_baseline     the CPU oracle's ingest on the host, GB/s
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
METRIC = "KV ingest GB/s (%HBM peak); added TTFT vs HBM-resident KV, 4K/64K prefix"


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


def setup(wl, log_every=8):
    import torch
    import kvgen
    import paper_2605_22850_amd as oc

    L, nq, nkv, d = wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    layout = oc.Layout(L, nq, nkv, d, wl.page_size, wl.chunk_tokens, wl.pool_pages)
    t = time.time()
    pool = torch.zeros(layout.pool_elems, dtype=torch.int16, device="cuda")
    tables = kvgen.block_tables(wl.seed, [wl.pages_needed(r) for r in range(wl.n_requests)], wl.pool_pages)
    reqs, objs_all = [], []
    for r in range(wl.n_requests):
        tp, ts = wl.prefix_tokens[r], wl.suffix_tokens[r]
        n = wl.n_chunks(r)
        objs = kvgen.chunk_objects(wl.seed, r, L, n, wl.slice_elems, threads=16)    # [N][L][S/2]
        objs_all.append(objs)
        b = 2 * nkv * d * 2
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


def run_mode(oc, pool, layout, wl, reqs, mode, trials, **kw):
    ctx = oc.oc_context_create(pool, layout, mode, max(wl.prefix_tokens), max(wl.suffix_tokens), **kw)
    out = []
    try:
        for _ in range(trials):
            st = oc.oc_pipeline_run(ctx, reqs, wl.num_layers)
            out.append((oc.oc_pipeline_last_ms(ctx), st))
    finally:
        oc.oc_context_destroy(ctx)
    return out


def cpu_baseline(wl, objs_all, tables, budget_s):
    """The CPU oracle, as it stands, on a bounded sample of the same workload."""
    import oracle
    L, nq, nkv, d, G, Ps = (wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim, wl.chunk_tokens,
                            wl.page_size)
    objs, table = objs_all[0], tables[0]
    n = objs.shape[0]
    tp = wl.prefix_tokens[0]
    pool = np.zeros(oracle.pool_shape(1, wl.pool_pages, nkv, Ps, d), dtype=np.uint16)
    layers, secs = 0, 0.0
    while layers < L and (layers == 0 or secs < budget_s * 0.5):
        staging = np.ascontiguousarray(objs[:, layers, :]).reshape(-1)
        t = time.perf_counter()
        oracle.ingest_layer(staging, n, G, nkv, d, Ps, table, pool, 0)
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
    threads = len(os.sched_getaffinity(0))
    rows, flops, asecs = [], 0.0, 0.0
    step = max(1, ts // 64)
    cand = list(range(ts - 1, -1, -step))
    for i in cand:
        if asecs > budget_s * 0.5 and rows:
            break
        t = time.perf_counter()
        oracle.attention(q, k, v, kn, vn, rows=[i], threads=threads)
        asecs += time.perf_counter() - t
        rows.append(i)
        flops += 4.0 * nq * d * (tp + i + 1)
    return {
        "value": round(ingest_gbs, 4), "unit": "GB/s", "cores": 1, "kind": "oracle",
        "sample": f"oracle byte-loop ingest of {layers} of {L} layers of request 0 ({layers * tp} tokens); "
                  f"the oracle's single-threaded scatter",
        "attention": {"gflops": round(flops / asecs / 1e9, 4), "threads": threads, "rows": len(rows),
                      "sample": f"float64 attention of {len(rows)} suffix rows x {nq} heads of layer 0 over "
                                f"{tp} prefix keys"},
        "seconds": round(secs + asecs, 2),
    }


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
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    args = ap.parse_args()

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the path has no cross-GPU part (see DESIGN.md for how it would "
              "shard); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import kvgen
    import paper_2605_22850_amd as oc

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    torch.cuda.set_device(0)
    wl = kvgen.workload(args.workload)
    L, nq, nkv, d = wl.num_layers, wl.num_q_heads, wl.num_kv_heads, wl.head_dim
    b = 2 * nkv * d * 2
    layout, pool, reqs, objs_all, tables = setup(wl)

    # ---- timed steps: device-staged pipeline, all layers ----
    for i in range(args.warmup):
        run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_DEVICE_STAGED, 1)
        log(f"[bench] warmup {i + 1}/{args.warmup}")
    ctx = oc.oc_context_create(pool, layout, oc.OC_MODE_DEVICE_STAGED, max(wl.prefix_tokens),
                               max(wl.suffix_tokens))
    ingest_ms, stage_ms, stats_all = 0.0, [], []
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        st = oc.oc_pipeline_run(ctx, reqs, L)
        stats_all.append(st)
        stage_ms.append(oc.oc_pipeline_last_ms(ctx))
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    oc.oc_context_destroy(ctx)
    log(f"[bench] {args.steps} steps in {wall:.3f} s")
    n_ingest = 0
    for st in stats_all:
        for rst in st:
            for l in range(L):
                ingest_ms += rst["ingested_ms"][l] - rst["landed_ms"][l]
                n_ingest += 1
    ingest_bytes_per_step = 2.0 * sum(wl.prefix_tokens) * b * L       # read + write, every layer
    value = ingest_bytes_per_step * args.steps / (ingest_ms / 1e3) / 1e9
    per_launch_bytes = 2.0 * sum(wl.prefix_tokens) * b / wl.n_requests
    mean_launch_us = ingest_ms / n_ingest * 1e3

    # ---- TTFT modes ----
    trials = max(2, args.trials)
    hbm = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_HBM_RESIDENT, trials)
    log("[bench] hbm-resident trials done")
    dev = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_DEVICE_STAGED, trials)
    log("[bench] device-staged trials done")
    t_hbm = [x[0] for x in hbm[1:]]
    t_dev = [x[0] for x in dev[1:]]
    # attention: per-layer compute of the attention-only pass
    total_flops = sum(attn_flops(nq, d, wl.prefix_tokens[r], wl.suffix_tokens[r]) for r in range(wl.n_requests)) * L
    attn_tflops = total_flops / (sum(t_hbm) / len(t_hbm) / 1e3) / 1e12
    ttft = {"hbm_resident": mean_std(t_hbm), "device_staged": mean_std(t_dev)}
    res = {}
    if not args.no_producer:
        unc = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials, rate_bytes_per_s=0.0)
        log("[bench] producer uncapped trials done")
        cap = run_mode(oc, pool, layout, wl, reqs, oc.OC_MODE_PRODUCER, trials, rate_bytes_per_s=args.cap)
        log("[bench] producer capped trials done")
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
    gates = {"device_staged_over_hbm": round((ttft["device_staged"][0] - ttft["hbm_resident"][0]) /
                                             ttft["hbm_resident"][0], 4)}

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(wall / args.steps * 1e3, 3), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic: seeded N(0,1) bf16 KV/Q, Fisher-Yates block tables",
        "config": {"workload": wl.name, "layers": L, "q_heads": nq, "kv_heads": nkv, "head_dim": d,
                   "prefix_tokens": wl.prefix_tokens if wl.n_requests > 1 else wl.prefix_tokens[0],
                   "suffix_tokens": wl.suffix_tokens if wl.n_requests > 1 else wl.suffix_tokens[0],
                   "page_tokens": wl.page_size, "chunk_tokens": wl.chunk_tokens, "pool_pages": wl.pool_pages,
                   "step": "device-staged pipeline: per layer ingest (copy stream) then attention (compute "
                           "stream), all layers"},
        "roofline": {"bound": "hbm", "kernel": "kv_ingest_kernel", "achieved": round(value, 2),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(value / HBM_PEAK_GBS, 4),
                     "traffic": None, "bytes_per_launch": per_launch_bytes,
                     "mean_launch_us": round(mean_launch_us, 3)},
        "attention": {"tflops": round(attn_tflops, 2), "peak": BF16_PEAK_TFLOPS,
                      "frac": round(attn_tflops / BF16_PEAK_TFLOPS, 4),
                      "flops_per_layer": total_flops / L,
                      "ms_per_layer": round(ttft["hbm_resident"][0] / L, 4)},
        "ttft_ms": ttft, **res, "gates": gates,
        "device_staged_ms": mean_std(stage_ms),
    }
    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle) ...")
        line["cpu_baseline"] = cpu_baseline(wl, objs_all, tables, args.cpu_budget)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
