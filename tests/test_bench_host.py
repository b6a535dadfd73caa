"""Host logic of bench.py on the CPU: the one-GPU guard, the simulator leg's
JSON line, and the algorithmic byte and flop counts behind the roofline
fractions, checked against per-row brute force; the committed chunk sweep
against its own points."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
import workload as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=300, cwd=ROOT)


def test_more_than_one_gpu_is_refused():
    r = run_bench("--gpus", "2")
    assert r.returncode == 2
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert "one GPU" in line["error"]


def test_simulate_prints_one_attainment_line():
    r = run_bench("--config", "c4", "--simulate",
                  os.path.join(ROOT, "profiles", "latency_model_layer_step_c4.json"),
                  "--rates", "4", "16", "--requests", "60")
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["rates"] == [4.0, 16.0]
    assert len(line["attainment"]) == 2
    for row in line["attainment"]:
        assert row["requests"] == 60
        assert 0.0 <= row["attainment"] <= 1.0
        assert row["ttft_p50_us"] <= row["ttft_p90_us"]
        assert row["tpot_p50_us"] <= row["tpot_p90_us"]


def brute_attention(cfg, b):
    """Flops and bytes of the attention, one query row at a time: a row at
    position p scores and weighs keys 0 .. p (4 nq d flops per key: q.k and
    p v, two flops per multiply-add); a decode row reads its request's keys
    and values and page table once; a prefill request reads each of its keys
    and values once (the chunk's own new keys included); every row reads its
    q and writes its o in bf16."""
    nq, d = cfg.n_q_heads, cfg.head_dim
    flops = 0.0
    dec_bytes = 0.0
    pre_bytes = 0.0
    for r in range(b.R):
        ctx, n = int(b.ctx_len[r]), int(b.n_new[r])
        for i in range(n):
            flops += 4.0 * nq * d * (ctx + i + 1)
        keys = ctx + n
        if b.phase[r] == wl.DECODE:
            dec_bytes += keys * cfg.kv_bytes_per_token + 2 * 2 * nq * d + 4 * -(-keys // 16)
        else:
            pre_bytes += keys * cfg.kv_bytes_per_token + n * 2 * 2 * nq * d
    return flops, dec_bytes, pre_bytes


def test_algorithmic_counts_match_brute_force():
    rng = np.random.default_rng(7)
    for key in ("c1", "c4"):
        cfg = wl.CONFIGS[key]
        b = wl.custom_batch(rng, [1, 15, 16, 17, 300], [(37, 0), (5, 40), (64, 1000)])
        parts = bench.algorithmic(cfg, b)
        flops, dec_bytes, pre_bytes = brute_attention(cfg, b)
        a = parts["attention"]
        assert a["flops"] == flops
        assert a["decode_bytes"] == dec_bytes
        assert a["bytes"] == dec_bytes + pre_bytes
        T, H, F = b.T, cfg.hidden, cfg.ffn
        nqd = cfg.n_q_heads * cfg.head_dim
        qkv = nqd + 2 * cfg.n_kv_heads * cfg.head_dim
        # each projection: 2 M N K flops; weights, input rows and output rows
        # once (bf16), plus the residual rows of the O and down projections
        for name, (N, K, n_out, res) in {"qkv": (qkv, H, qkv, 0), "o": (H, nqd, H, 1),
                                         "gate_up": (2 * F, H, F, 0),
                                         "down": (H, F, H, 1)}.items():
            assert parts[name]["flops"] == 2.0 * T * N * K
            assert parts[name]["bytes"] == 2.0 * (N * K + T * K + T * n_out) + res * 2.0 * T * N


def test_committed_chunk_sweep_follows_from_its_points():
    """profiles/chunk_sweep_layer_step_c4.json: chunk k continues a prompt with
    k chunks cached; its prefill attention flops are the per-row sum over the
    chunk's rows, and both recorded line fits refit from the recorded points."""
    rec = json.load(open(os.path.join(ROOT, "profiles", "chunk_sweep_layer_step_c4.json")))
    sw = rec["chunk_sweep"]
    cfg = wl.CONFIGS["c4"]
    C = sw["chunk"]
    pts = sw["points"]
    for p in pts:
        assert p["ctx"] == p["k"] * C and p["T"] == 256 + C
        rows = p["ctx"] + np.arange(C, dtype=np.float64)  # positions of the chunk's rows
        assert p["prefill_attn_flops"] == float((4.0 * cfg.n_q_heads * cfg.head_dim * (rows + 1)).sum())
    k = np.array([p["k"] for p in pts], dtype=np.float64)
    for field, fit in (("us", sw["fit_us_per_chunk_index"]),
                       ("attn_us", sw["fit_attention_us_per_chunk_index"])):
        y = np.array([p[field] for p in pts])
        slope, icpt = np.polyfit(k, y, 1)
        r2 = 1.0 - ((y - (slope * k + icpt)) ** 2).sum() / ((y - y.mean()) ** 2).sum()
        assert fit["points"] == len(pts)
        assert slope == pytest.approx(fit["slope_us_per_chunk_index"], abs=1e-3)
        assert icpt == pytest.approx(fit["intercept_us"], abs=1e-2)
        assert r2 == pytest.approx(fit["r2"], abs=1e-4)


def test_committed_traffic_summaries_are_consistent():
    """Every profiles/traffic_*.json: the copy calibration scales the counters
    (bytes of the 1 GiB copy over what each counter read for it), the per-launch
    bytes are the scaled counter means, and the algorithmic bytes beside them
    are the kernel's part of the workload it names."""
    paths = sorted(p for p in os.listdir(os.path.join(ROOT, "profiles"))
                   if p.startswith("traffic_") and p.endswith(".json"))
    assert paths
    for name in paths:
        rec = json.load(open(os.path.join(ROOT, "profiles", name)))
        cal = rec["copy_calibration"]
        fs = cal["bytes"] / (cal["FETCH_SIZE_KiB"] * 1024.0)
        ws = cal["bytes"] / (cal["WRITE_SIZE_KiB"] * 1024.0)
        assert cal["fetch_scale"] == pytest.approx(fs, abs=1e-4)
        assert cal["write_scale"] == pytest.approx(ws, abs=1e-4)
        # the recorded means are rounded to 0.1 KiB
        fetch = rec["FETCH_SIZE_KiB_mean"] * 1024.0 * fs
        write = rec["WRITE_SIZE_KiB_mean"] * 1024.0 * ws
        assert rec["fetch_bytes_per_launch"] == pytest.approx(fetch, abs=0.05 * 1024 * fs + 1)
        assert rec["write_bytes_per_launch"] == pytest.approx(write, abs=0.05 * 1024 * ws + 1)
        assert rec["hbm_bytes_per_launch"] == pytest.approx(
            rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"], abs=1)
        key, P = rec["workload"].split("_P")
        part, _ = bench.TRAFFIC_TAGS[rec["tag"]]
        parts = bench.algorithmic(wl.CONFIGS[key], wl.make_batch(key, int(P)))
        assert rec["algorithmic_bytes_per_launch"] == int(parts[part]["bytes"])


def test_too_few_predictor_batches_are_refused_before_any_gpu_work():
    r = run_bench("--predictor", "4")
    assert r.returncode != 0
    assert "at least 12" in r.stderr
