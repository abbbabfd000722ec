"""Host-side logic of bench.py, no GPU: the one-GPU guard, the eq. (3) and
chunkwise floors it reports beside the measured TTFT (against the oracle's
model), the attention FLOP count (against a brute-force count of the
unmasked query-key pairs), and the arithmetic that turns rocprofv3 counter
databases into the HBM-traffic figure (on a synthetic database)."""
import json
import os
import sqlite3
import subprocess
import sys

import numpy as np
import pytest

import bench
from oracle import model

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("argv,env", [(["--gpus", "2"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(argv, env):
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *argv], capture_output=True, text=True,
                       env={**os.environ, **env}, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout.strip()


def test_floors_match_the_oracle_model():
    rng = np.random.default_rng(3)
    for L in (1, 2, 5, 32):
        X, C = rng.uniform(0, 2, L).tolist(), rng.uniform(0, 2, L).tolist()
        assert bench.layerwise_floor(X, C) == pytest.approx(model.layerwise_ttft(X, C), rel=1e-12)
        assert bench.chunkwise_floor(X, C) == pytest.approx(model.chunkwise_ttft(X, C), rel=1e-12)


@pytest.mark.parametrize("tp,ts", [(0, 1), (0, 7), (16, 1), (256, 32), (100, 13)])
def test_attention_flops_count_unmasked_pairs(tp, ts):
    nq, d = 4, 64
    pairs = sum(1 for i in range(ts) for j in range(tp + ts) if j < tp or j - tp <= i)
    assert bench.attn_flops(nq, d, tp, ts) == 4 * nq * d * pairs


def _counter_db(path, counter, calib_kib, ingest_kib, n_ingest):
    """A database with the columns the summary reads: three 1 GiB calibration
    copies, then n_ingest ingest dispatches, each with one counter value."""
    c = sqlite3.connect(path)
    c.execute("create table counters_collection (dispatch_id int, kernel_name text, counter_name text, "
              "value real, start int, end int)")
    t = 1000
    rows = []
    for i in range(bench.CALIB_COPIES):
        rows.append((i, "__amd_rocclr_copyBuffer", counter, calib_kib, t, t + 300000))
        t += 400000
    for i in range(n_ingest):
        rows.append((100 + i, "oc::kv_ingest_rows_kernel", counter, ingest_kib, t, t + 100000))
        t += 200000
    c.executemany("insert into counters_collection values (?,?,?,?,?,?)", rows)
    c.commit()
    c.close()


def test_profile_summary_scales_the_byte_counters(tmp_path):
    # tiny: 2 layers, one request -> 2 ingest launches per run; warmup 1, steps 2
    # select launches 2..5.  Calibration reads half the copied bytes, so the
    # scale is 2 for FETCH_SIZE; WRITE_SIZE reads them exactly (scale 1).
    expect = bench.CALIB_COPIES * bench.CALIB_BYTES / 1024.0
    f, w = str(tmp_path / "pf.db"), str(tmp_path / "pw.db")
    _counter_db(f, "FETCH_SIZE", expect / bench.CALIB_COPIES / 2, 100.0, 8)
    _counter_db(w, "WRITE_SIZE", expect / bench.CALIB_COPIES, 128.0, 8)
    text = bench.profile_summary([f, w], "tiny", 1, 2)
    want = 100.0 * 1024 * 2 + 128.0 * 1024
    line = [ln for ln in text.splitlines() if ln.startswith("traffic_bytes_per_launch:")]
    assert line and float(line[0].split(":")[1]) == pytest.approx(want, rel=1e-9)
    assert f"kernel_source_sha256: {bench.file_sha256(bench.INGEST_SRC)}" in text
    # the algorithmic bytes of a tiny layer: 256 tokens x 512 B, read + written
    assert "Algorithmic bytes per launch: 262144" in text


def test_cpu_baseline_reports_its_sample():
    import kvgen
    wl = kvgen.workload("tiny")
    objs = kvgen.chunk_objects(wl.seed, 0, wl.num_layers, wl.n_chunks(0), wl.slice_elems)
    tables = kvgen.block_tables(wl.seed, [wl.pages_needed(0)], wl.pool_pages)
    r = bench.cpu_baseline(wl, [objs], tables, 1.0)
    assert r["kind"] == "oracle" and r["value"] > 0 and r["cpu"] and r["cpu"] != "unknown"
    assert r["cores"] == min(16, len(os.sched_getaffinity(0)))
    a = r["attention"]
    assert a["rows"] == wl.suffix_tokens[0] and a["gflops"] > 0
    assert a["all_layers_s_extrapolated"] == pytest.approx(wl.num_layers * a["layer_s_extrapolated"], abs=0.1)


def test_cells_summary_formats_sweep_and_sensitivity(tmp_path):
    cell = {"context": 65536, "hit": 0.5, "prefix_tokens": 32768, "suffix_tokens": 32768,
            "compute_ms_per_layer": 35.0, "transfer_ms_per_layer_at_cap": 10.7, "layer_tflops": 1100.0,
            "ttft_ms": {"hbm_resident": 1130.0, "producer_uncapped": 1140.0, "capped_layerwise": 1150.0,
                        "capped_chunkwise": 1480.0},
            "eq3_ms": 1146.0, "chunkwise_model_ms": 1479.0, "added_over_hbm_pct": {"capped_layerwise": 1.77},
            "required_GBps": 3.83,
            "rate_sweep": [{"rate_GBps": 1.25, "layerwise_ms": 3470.0, "chunkwise_ms": 4580.0, "eq3_ms": 3468.0,
                            "chunkwise_model_ms": 4570.0},
                           {"rate_GBps": 12.5, "layerwise_ms": 1150.0, "chunkwise_ms": 1480.0, "eq3_ms": 1146.0,
                            "chunkwise_model_ms": 1479.0}],
            "bandwidth_sensitivity": bench.bandwidth_sensitivity(
                [{"rate_GBps": 1.25, "layerwise_ms": [3470.0], "chunkwise_ms": [4580.0]},
                 {"rate_GBps": 12.5, "layerwise_ms": [1150.0], "chunkwise_ms": [1480.0]}])}
    p = tmp_path / "cells.json"
    p.write_text("noise\n" + json.dumps({"canonical_cells": {"cap_GBps": 12.5, "chunk_tokens": 64, "ffn_dim": 14336,
                                                             "cells": [cell]}}) + "\n")
    text = bench.cells_summary(str(p))
    assert "| 64K | 50 % | 32768 / 32768 | 35.0 | 10.7 |" in text
    assert "| 64K | 50 % | 3.83 | 1.25 | 3470.0 | 3468.0 | 1.001 |" in text
    # 3470 / 1150 - 1 and 4580 / 1480 - 1
    assert "| 64K | 50 % | 3.83 | +201.7 % | +209.5 % |" in text


def test_marker_summary_splits_each_layers_delivery(tmp_path):
    # one run, two layers: marks at 1000 and 3000 ns; layer 0 lands in two
    # spans (ending 1500 and 2000) and is ingested at 2100, layer 1 in one
    # span (ending 3500), ingested at 3600
    db = tmp_path / "m.db"
    c = sqlite3.connect(db)
    c.execute("create table regions (extdata text, tid int, start int, end int)")
    c.execute("create table samples (extdata text, tid int, timestamp int)")
    c.execute("create table kernels (name text, start int, end int)")
    c.execute("create table memory_copies (start int, end int, size int, src_agent_type text)")
    msg = lambda m: json.dumps({"message": m})  # noqa: E731
    c.executemany("insert into regions values (?,?,?,?)",
                  [(msg("oc_pipeline_run"), 7, 0, 100000), (msg("layer 0 req 0"), 7, 10, 2050),
                   (msg("layer 1 req 0"), 7, 2060, 3550), (msg("layer 0 req 0"), 8, 20, 30)])
    c.executemany("insert into samples values (?,?,?)", [(msg("ready layer 0 req 0"), 9, 1000),
                                                         (msg("ready layer 1 req 0"), 9, 3000)])
    c.executemany("insert into kernels values (?,?,?)",
                  [("oc::kv_ingest_src_kernel<true>", 2100, 2200), ("oc::attn_fwd_kernel<128>", 2200, 2900),
                   ("oc::kv_ingest_rows_kernel", 3600, 3700)])
    c.executemany("insert into memory_copies values (?,?,?,?)",
                  [(1000, 1500, 1000, "CPU"), (1500, 2000, 1000, "CPU"), (3000, 3500, 1000, "CPU"),
                   (50000, 50100, 99, "GPU")])
    c.commit()
    c.close()
    out = bench.marker_summary([str(db)])
    assert "| range | `layer` | 3 |" in out and "| mark | `ready` | 2 |" in out
    row = next(ln for ln in out.splitlines() if ln.startswith("| 0 |"))
    cells = [x.strip() for x in row.strip("|").split("|")]
    # run, host ms, layer ranges (driver thread only), mean range us, marks, mark gap ms,
    # spans per layer, DMA GB/s, mark -> last span, last span -> ingest, mark -> ingest (max)
    assert cells == ["0", "0.10", "2", "1.8", "2", "0.002", "1.5", "2.0", "0.8", "0.1", "0.8 (1.1)"]


def test_step_ingest_counts_a_shared_launch_once():
    # two requests of two layers, 400 tokens of 32 bytes per layer: 51200
    # bytes read + written per run; layer 0 ingested by one launch for both
    # (the same marker pair), layer 1 by one launch each
    class W:
        num_layers, num_kv_heads, head_dim, prefix_tokens = 2, 1, 8, [100, 300]
    runs = [[{"landed_ms": [0.0, 2.0], "ingested_ms": [1.0, 2.5]},
             {"landed_ms": [0.0, 2.5], "ingested_ms": [1.0, 3.5]}]]
    r = bench.step_ingest(runs, W)
    assert r["launches"] == 3
    assert r["mean_launch_us"] == pytest.approx(2500.0 / 3)
    assert r["value"] == pytest.approx(round(51200 / 2.5e-3 / 1e9, 2))
