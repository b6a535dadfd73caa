"""Benchmark of the multiplexed decoder-layer iteration on one MI355X.

A step is one mx_layer_step over one mixed batch (prefill chunks co-batched
with decodes): token map, RMSNorm, QKV GEMM, RoPE + KV append, paged attention
(one launch for prefill and decode rows), O GEMM + residual, RMSNorm, gate/up
GEMM + SwiGLU, down GEMM + residual.  Inputs are synthetic, seeded, and
resident in HBM before the timed region.

Default workload: the 70B-shaped layer (hidden 8192, 64 query / 8 KV heads x
128, FFN 28672) with 256 decodes (contexts uniform in [1024, 16384], a KV pool
of about 150 GB) plus 0 .. 8192 mixed prefill tokens in steps of 1024; the
headline is the last point (8192 prefill tokens, T = 8448) and the whole sweep
is the latency-vs-mixed-prefill curve.  `--config c2|c3|c4` times the other
shapes.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "mixed-batch layer iteration latency (µs) & tokens/s vs prefill tokens mixed"
HBM_PEAK = 8.0e12        # bytes/s, MI355X
MFMA_BF16_PEAK = 2.5e15  # flop/s, dense bf16


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=int(os.environ.get("WORLD_SIZE", "1")))
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=100)
    ap.add_argument("--config", default="c5", help="layer shape c1..c5")
    ap.add_argument("--prefill", type=int, nargs="*", default=None,
                    help="mixed prefill tokens per point (default: the shape's sweep)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle CPU baseline")
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--kernels", action="store_true", default=True)
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="run one plain device copy of this many MiB before timing (the "
                         "known-size reference that scales rocprofv3 byte counters)")
    ap.add_argument("--chunk-sweep", nargs=2, type=int, metavar=("CHUNK", "N"),
                    help="chunk-index sweep: the shape's decode batch plus one CHUNK-token "
                         "prefill chunk continuing a prompt with k*CHUNK tokens cached, "
                         "k = 0..N-1; prints one JSON line with latency per chunk index")
    ap.add_argument("--predictor", type=int, metavar="N",
                    help="time N random batches of the shape (random decode count and "
                         "contexts, random chunk length and prior context), fit the linear "
                         "latency model on the even-numbered ones and report its residuals "
                         "on the odd-numbered ones; prints one JSON line")
    ap.add_argument("--simulate", metavar="MODEL_JSON",
                    help="CPU only: SLO attainment of SLO-aware multiplexed serving over a sweep "
                         "of arrival rates, simulated with the "
                         "latency model that `--predictor` printed (MODEL_JSON); prints one JSON line")
    ap.add_argument("--rates", type=float, nargs="+", default=[4, 8, 16, 24, 32, 48])
    ap.add_argument("--requests", type=int, default=800)
    ap.add_argument("--summarize-stats", nargs=4,
                    metavar=("STATS_CSV", "COMMAND", "WORKLOAD", "OUT_MD"),
                    help="write a markdown summary of a rocprofv3 --stats kernel_stats.csv of "
                         "the step on WORKLOAD (e.g. c5_P8192) (no GPU needed)")
    ap.add_argument("--summarize-traffic", nargs="+",
                    metavar="ARG",
                    help="FETCH_CSV WRITE_CSV COMMANDS_TXT WORKLOAD OUT_JSON [TAG KERNEL_NAME]: "
                         "HBM bytes per launch of one kernel of the step (default: the attention; "
                         "TAG a step tag such as gemm_gate_up and KERNEL_NAME the exact kernel "
                         "name prefix in the trace) from two rocprofv3 --pmc runs (FETCH_SIZE, "
                         "WRITE_SIZE), scaled by the 1 GiB copy calibration they contain "
                         "(no GPU needed)")
    return ap.parse_args()


def workload_text(workload):
    """One line describing a sweep point such as c5_P8192."""
    import workload as wl
    key, P = workload.split("_P")
    cfg = wl.CONFIGS[key]
    b = wl.make_batch(key, int(P))
    n_dec = int((b.phase == wl.DECODE).sum())
    return (f"{cfg.name}-shaped layer: hidden {cfg.hidden}, {cfg.n_q_heads} query / "
            f"{cfg.n_kv_heads} KV heads x {cfg.head_dim}, FFN {cfg.ffn}; {n_dec} decodes "
            f"(contexts {int(b.ctx_len[b.phase == wl.DECODE].min())}.."
            f"{int(b.ctx_len[b.phase == wl.DECODE].max())}) with {b.prefill_tokens} mixed prefill "
            f"tokens, T = {b.T}")


def summarize_stats(csv_path, command, workload, out_md):
    """Markdown table of a rocprofv3 --kernel-trace --stats summary."""
    import csv
    rows = list(csv.DictReader(open(csv_path)))
    total = sum(float(r["TotalDurationNs"]) for r in rows)
    lines = [f"# Kernel trace statistics: the layer step, {workload}", "",
             f"Workload: {workload_text(workload)}.  The run includes setup (weight packing, pool "
             "fill) and the per-kernel timing steps.", "",
             "Command (one MI355X):", "", "```", command, "```", "",
             "Durations in microseconds (rocprofv3 kernel trace).  gemm_kernel<BM, BN, WM, WN, LDS stages, "
             "epilogue, split>: epilogue 0 store, 1 residual, 2 SwiGLU, 3 QKV.", "",
             "| kernel | calls | average us | min us | max us | share % |",
             "|---|---:|---:|---:|---:|---:|"]
    rows.sort(key=lambda r: -float(r["TotalDurationNs"]))
    for r in rows:
        name = r["Name"].replace("(anonymous namespace)::", "").replace("mx::", "")
        name = name.split("(")[0].replace("void ", "")
        lines.append(f"| `{name}` | {r['Calls']} | {float(r['AverageNs']) / 1e3:.1f} | "
                     f"{float(r['MinNs']) / 1e3:.1f} | {float(r['MaxNs']) / 1e3:.1f} | "
                     f"{100.0 * float(r['TotalDurationNs']) / total:.1f} |")
    with open(out_md, "w") as f:
        f.write("\n".join(lines) + "\n")


# step tag -> (algorithmic part, source file of its kernel)
TRAFFIC_TAGS = {"paged_attn": ("attention", "paper_2606_16264_amd/csrc/attention.hip"),
                "gemm_qkv": ("qkv", "paper_2606_16264_amd/csrc/gemm.hip"),
                "gemm_o": ("o", "paper_2606_16264_amd/csrc/gemm.hip"),
                "gemm_gate_up": ("gate_up", "paper_2606_16264_amd/csrc/gemm.hip"),
                "gemm_down": ("down", "paper_2606_16264_amd/csrc/gemm.hip")}


def summarize_traffic(fetch_csv, write_csv, commands_txt, workload, out_json,
                      tag="paged_attn", kernel="paged_attn_kernel"):
    """HBM bytes per launch of `kernel` (the kernel of step `tag`):
    FETCH_SIZE and WRITE_SIZE (KiB per dispatch) scaled by what the same
    counters read for the 1 GiB device copy (torch's copyBuffer) recorded in
    the same runs."""
    part, source = TRAFFIC_TAGS[tag]
    import csv
    calib = 1 << 30

    def read(path, counter):
        ks, cp = [], []
        for r in csv.DictReader(open(path)):
            if r["Counter_Name"] != counter:
                continue
            v = float(r["Counter_Value"])
            name = r["Kernel_Name"].replace("(anonymous namespace)::", "").replace("mx::", "")
            name = name.replace("void ", "")
            if name.startswith(kernel):
                ks.append(v)
            elif "copyBuffer" in r["Kernel_Name"]:
                cp.append(v)
        return ks, max(cp)  # the calibration copy is the largest copy in the run
    kf, cf = read(fetch_csv, "FETCH_SIZE")
    kw, cw = read(write_csv, "WRITE_SIZE")
    fs, ws_ = calib / (cf * 1024.0), calib / (cw * 1024.0)
    fetch = sum(kf) / len(kf) * 1024.0 * fs
    write = sum(kw) / len(kw) * 1024.0 * ws_
    key, P = workload.split("_P")
    import workload as wl
    parts = algorithmic(wl.CONFIGS[key], wl.make_batch(key, int(P)))
    rec = {"kernel": kernel, "tag": tag, "workload": workload,
           "commands": [l.strip() for l in open(commands_txt) if l.strip()],
           "copy_calibration": {"bytes": calib, "FETCH_SIZE_KiB": cf, "WRITE_SIZE_KiB": cw,
                                "fetch_scale": round(fs, 4), "write_scale": round(ws_, 4)},
           "dispatches": len(kf), "FETCH_SIZE_KiB_mean": round(sum(kf) / len(kf), 1),
           "WRITE_SIZE_KiB_mean": round(sum(kw) / len(kw), 1),
           "fetch_bytes_per_launch": int(fetch), "write_bytes_per_launch": int(write),
           "hbm_bytes_per_launch": int(fetch + write),
           "algorithmic_bytes_per_launch": int(parts[part]["bytes"]),
           "source_sha256": source_sha(source)}
    with open(out_json, "w") as f:
        json.dump(rec, f, indent=1)


def source_sha(rel):
    import hashlib
    with open(os.path.join(ROOT, rel), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def measured_traffic(kernel, workload, source):
    """HBM bytes per launch of `kernel` on `workload` from the committed
    rocprofv3 counter summary (profiles/traffic_<kernel>_<workload>.json), or
    None when there is none or the kernel source changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != source_sha(source):
        return None
    return rec.get("hbm_bytes_per_launch")


def algorithmic(cfg, b):
    """Algorithmic bytes / flops of the iteration's parts (what the method must
    move or compute: no padding, K/V read once per KV head)."""
    import numpy as np
    import workload as wl
    H, F, nq, nkv, d = cfg.hidden, cfg.ffn, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    T = b.T
    KVB = cfg.kv_bytes_per_token
    gemms = {
        "qkv": (T, cfg.qkv_rows, H),
        "o": (T, H, nq * d),
        "gate_up": (T, 2 * F, H),
        "down": (T, H, F),
    }
    out = {}
    for name, (M, N, K) in gemms.items():
        n_out = N // 2 if name == "gate_up" else N
        res = M * N * 2 if name in ("o", "down") else 0
        out[name] = dict(flops=2.0 * M * N * K, bytes=2.0 * (N * K + M * K + M * n_out) + res)
    dec = b.phase == wl.DECODE
    ctx1 = (b.ctx_len[dec].astype(np.int64) + 1)
    dec_bytes = float((ctx1 * KVB).sum() + dec.sum() * 4 * nq * d
                      + (4 * np.ceil(ctx1 / 16)).sum())
    dec_flops = float((4 * nq * d * ctx1).sum())
    pre = ~dec
    p = b.ctx_len[pre].astype(np.int64)
    t = b.n_new[pre].astype(np.int64)
    pre_flops = float((4 * nq * d * (p * t + t * (t + 1) / 2)).sum())
    pre_bytes = float(((p + t) * KVB + 4 * t * nq * d).sum())
    out["attention"] = dict(flops=dec_flops + pre_flops, bytes=dec_bytes + pre_bytes,
                            decode_bytes=dec_bytes, prefill_flops=pre_flops)
    out["kv_append"] = dict(flops=0.0, bytes=2.0 * T * KVB)
    out["rmsnorm"] = dict(flops=0.0, bytes=8.0 * T * H)
    return out


def t_roof(parts):
    return sum(max(p["flops"] / MFMA_BF16_PEAK, p["bytes"] / HBM_PEAK) for p in parts.values())


class Point:
    """Device state of one sweep point."""

    def __init__(self, key, P, w_dev, packed, cfg, batch=None):
        import torch
        import paper_2606_16264_amd as mx
        import workload as wl
        import workload.device as wdev
        self.key, self.P, self.cfg = key, P, cfg
        self.b = batch if batch is not None else wl.make_batch(key, P)
        b = self.b
        self.c = mx.layer_cfg(cfg.hidden, cfg.ffn, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                              b.pool_pages, cfg.rms_eps, cfg.rope_theta)
        self.shape = self.c.attn
        self.packed = packed
        self.k, self.v = wdev.alloc_pools(cfg, b.pool_pages)
        wdev.fill_pools(self.k, self.v, cfg, b, wl.kv_seed(key), poison=True)
        self.mb = mx.Batch(b.phase, b.n_new, b.ctx_len, b.page_tables)
        self.ws = torch.empty(mx.mx_workspace_bytes_for(self.mb, cfg=self.c), dtype=torch.uint8,
                              device="cuda")
        self.x = torch.from_numpy(wl.make_x(cfg, b.T, key)).cuda()
        self.y = torch.empty_like(self.x)
        self.parts = algorithmic(cfg, b)

    def step(self):
        import paper_2606_16264_amd as mx
        mx.mx_layer_step(self.mb, self.c, self.packed, self.x, self.y, self.k, self.v, self.ws)

    def release(self):
        del self.k, self.v, self.ws


def time_fn(fn, steps, warmup):
    """Mean ms per step over `steps` back-to-back steps (events bracketing the
    whole run), plus the per-step distribution from events around each step,
    and the host's own time to plan and enqueue one step (taken over the first
    calls after a synchronisation, before the library's ring of eight staging
    buffers can make the host wait for the device)."""
    import time
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    n_host, host_ms = min(steps, 6), 0.0
    s.record()
    t0 = time.perf_counter()
    for i in range(steps):
        fn()
        if i == n_host - 1:
            host_ms = (time.perf_counter() - t0) * 1e3 / n_host
    e.record()
    torch.cuda.synchronize()
    mean = s.elapsed_time(e) / steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    ev[0].record()
    for i in range(steps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = sorted(ev[i].elapsed_time(ev[i + 1]) for i in range(steps))

    def q(f):
        return per[min(len(per) - 1, int(round(f * (len(per) - 1))))]
    return mean, {"median": q(0.5), "p10": q(0.1), "p90": q(0.9), "host": host_ms}


def linear_fit(xs, ys, slope_name="slope_us_per_prefill_token"):
    """Least-squares line y = a + b x with R^2 (the latency-vs-prefill curve)."""
    n = len(xs)
    if n < 2:
        return None
    mx_, my = sum(xs) / n, sum(ys) / n
    sxx = sum((x - mx_) ** 2 for x in xs)
    if sxx == 0:
        return None
    b = sum((x - mx_) * (y - my) for x, y in zip(xs, ys)) / sxx
    a = my - b * mx_
    ss_tot = sum((y - my) ** 2 for y in ys)
    ss_res = sum((y - a - b * x) ** 2 for x, y in zip(xs, ys))
    return {"intercept_us": round(a, 2), slope_name: round(b, 5),
            "r2": round(1.0 - ss_res / ss_tot, 5) if ss_tot > 0 else 1.0, "points": n}


def kernel_breakdown(pt, steps, warmup):
    """Per-kernel durations of the step's own launches, measured live with the
    library's launch timing (hipEvents recorded on the launch stream around
    each kernel), with each part's algorithmic roofline fraction."""
    import paper_2606_16264_amd as mx
    for _ in range(warmup):
        pt.step()
    mx.mx_profile_read()
    mx.mx_profile_enable(True)
    for _ in range(steps):
        pt.step()
    mx.mx_profile_enable(False)
    times = mx.mx_profile_read()
    parts = pt.parts
    # the second RMSNorm runs fused with the output projection's split-K reduce
    # when (some rows of) that projection are split over K: it then also reads
    # the fp32 planes and the residual of the split rows and writes their x1
    cfg, T = pt.cfg, pt.b.T
    plan = mx.mx_debug_gemm_plan(T, cfg.hidden, cfg.n_q_heads * cfg.head_dim)
    split_rows = T - plan["m_main"] if plan["m_main"] < T else T
    ks = plan["tail_ksplit"] if plan["m_main"] < T else plan["ksplit"]
    norm2 = parts["rmsnorm"]["bytes"] / 2
    fused = norm2 + split_rows * cfg.hidden * (4.0 * ks + 2.0 + 2.0)
    algo = {"gemm_qkv": parts["qkv"], "gemm_o": parts["o"], "gemm_gate_up": parts["gate_up"],
            "gemm_down": parts["down"], "paged_attn": parts["attention"],
            "token_map+rmsnorm_1": {"flops": 0.0, "bytes": parts["rmsnorm"]["bytes"] / 2},
            "rmsnorm_2": {"flops": 0.0, "bytes": norm2},
            "o_reduce+rmsnorm_2": {"flops": 0.0, "bytes": fused}}
    res = {}
    for tag, (ms, n) in times.items():
        us = ms / max(n, 1) * 1e3
        a = algo.get(tag, {"flops": 0.0, "bytes": 0.0})
        sec = us * 1e-6
        res[tag] = dict(us=us, launches=n, flops=a["flops"], bytes=a["bytes"],
                        hbm_frac=a["bytes"] / sec / HBM_PEAK if sec > 0 else 0.0,
                        mfma_frac=a["flops"] / sec / MFMA_BF16_PEAK if sec > 0 else 0.0,
                        achieved_GBps=a["bytes"] / sec / 1e9 if sec > 0 else 0.0,
                        TFLOPs=a["flops"] / sec / 1e12 if sec > 0 else 0.0)
    return res


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(key, cfg, w_host, budget_s):
    """The fp64 oracle (as it stands) on a bounded sample of the same workload:
    a sub-batch of decode requests plus the first tokens of the prefill chunk,
    every row evaluated.  Reported as tokens/s on the host cores."""
    import numpy as np
    import oracle
    import workload as wl
    b = wl.make_batch(key, max(wl.SWEEPS[key]))
    x = wl.make_x(cfg, b.T, key)
    seed = wl.kv_seed(key)
    dec = [r for r in range(b.R) if b.phase[r] == wl.DECODE]
    pre = [r for r in range(b.R) if b.phase[r] == wl.PREFILL]
    start = np.concatenate([[0], np.cumsum(b.n_new)])

    def run(n_dec, n_pre_tok):
        reqs = dec[:n_dec] + pre[:1]
        sub = b.subset(reqs)
        if pre:
            sub.n_new[-1] = min(n_pre_tok, int(sub.n_new[-1]))
        tok = []
        for i, r in enumerate(reqs):
            tok += list(range(int(start[r]), int(start[r]) + int(sub.n_new[i])))
        kp, vp = wl.prior_kv_concat(cfg, sub, seed)
        t0 = time.perf_counter()
        oracle.layer_step(cfg.as_dict(), sub.n_new, sub.ctx_len, x[tok], w_host, kp, vp)
        return time.perf_counter() - t0, sub.T

    # grow the sample until one evaluation takes about the requested budget
    n_dec, n_pre = 2, 2
    dt, n = run(n_dec, n_pre)
    while dt < budget_s / 2 and (n_dec < len(dec) or (pre and n_pre < int(b.n_new[pre[0]]))):
        grow = min(4.0, max(1.5, budget_s / max(dt, 1e-3) / 1.5))
        n_dec = int(min(len(dec), max(n_dec + 1, round(n_dec * grow))))
        n_pre = int(max(n_pre + 1, round(n_pre * grow)))
        dt, n = run(n_dec, n_pre)
    # the whole batch fits the budget: repeat it until the budget is spent
    reps, total = 1, dt
    while total < budget_s / 2:
        dt2, _ = run(n_dec, n_pre)
        total += dt2
        reps += 1
    return {"value": n * reps / total, "unit": "tokens/s", "cores": oracle.num_threads(),
            "kind": "oracle",
            "sample": f"{n_dec} decode requests + first {n_pre} tokens of the prefill chunk "
                      f"({n} rows, full layer), {reps} evaluation(s) in {total:.1f} s",
            "oracle": "plain C, fp64 arithmetic, gcc " + " ".join(oracle.CFLAGS),
            "cpu": cpu_model()}


def chunk_sweep(args, key, cfg, packed):
    """Latency of the step as the same chunk moves later in its prompt: chunk
    k attends over k * CHUNK cached tokens plus its own causal triangle, so its
    attention work grows linearly with k while the projections stay fixed."""
    import numpy as np
    import workload as wl
    C, N = args.chunk_sweep
    b0 = wl.make_batch(key, 0)
    dec_ctx = [int(c) for c in b0.ctx_len]
    pts = []
    for k in range(N):
        b = wl.make_batch(key, C, decode_ctx=dec_ctx, prefill_lens=[C], prefill_ctx=[k * C])
        pt = Point(key, C, None, packed, cfg, batch=b)
        ms, dist = time_fn(pt.step, args.steps, args.warmup)
        kern = kernel_breakdown(pt, max(5, args.steps // 2), 2)
        rec = dict(k=k, ctx=k * C, T=b.T, us=round(ms * 1e3, 2), us_median=round(dist["median"] * 1e3, 2),
                   attn_us=round(kern["paged_attn"]["us"], 2),
                   prefill_attn_flops=pt.parts["attention"]["prefill_flops"],
                   t_roof_us=round(t_roof(pt.parts) * 1e6, 2))
        print(f"# chunk {k}: ctx {k * C}: {rec['us']} us (attention {rec['attn_us']} us)",
              file=sys.stderr, flush=True)
        pts.append(rec)
        pt.release()
    fit = linear_fit([p["k"] for p in pts], [p["us"] for p in pts], "slope_us_per_chunk_index")
    fit_attn = linear_fit([p["k"] for p in pts], [p["attn_us"] for p in pts], "slope_us_per_chunk_index")
    print(json.dumps({"chunk_sweep": {"workload": f"{cfg.name} layer ({key}): "
                                                  f"{int(b0.R)} decodes + one {C}-token chunk",
                                      "chunk": C, "points": pts,
                                      "fit_us_per_chunk_index": fit,
                                      "fit_attention_us_per_chunk_index": fit_attn}}))


def predictor_batches(key, n):
    """The random batches the latency model is fitted on, in order (seeded):
    (record, batch) with 8-256 decodes at contexts U[64, 4096] and a chunk of
    0-4096 tokens after 0-4096 cached ones."""
    import numpy as np
    import workload as wl
    rng = np.random.default_rng(2024)
    max_dec = 256
    for _ in range(n):
        n_dec = int(rng.integers(8, max_dec + 1))
        dec_ctx = [int(c) for c in rng.integers(64, 4097, size=n_dec)]
        P = int(rng.choice([0, 0, 128, 512, 1024, 2048, 4096]))
        pctx = int(rng.choice([0, 0, 1024, 4096])) if P else 0
        b = wl.make_batch(key, P, decode_ctx=dec_ctx, prefill_lens=[P] if P else [],
                          prefill_ctx=[pctx] if P else [])
        yield dict(n_decode=n_dec, P=P, prefill_ctx=pctx, T=int(b.T)), b


def predictor_fit(args, key, cfg, packed):
    """Fit of the iteration-latency model to measured steps of random batches
    (held-out residuals test how predictable the mixed iteration is)."""
    import workload as wl
    from paper_2606_16264_amd.sched import LatencyModel, batch_features
    feats, lat, recs = [], [], []
    for i, (rec, b) in enumerate(predictor_batches(key, args.predictor)):
        P = rec["P"]
        pt = Point(key, P, None, packed, cfg, batch=b)
        ms, _ = time_fn(pt.step, args.steps, args.warmup)
        f = batch_features(b.n_new, b.ctx_len, b.phase == wl.DECODE)
        feats.append(f)
        lat.append(ms * 1e3)
        recs.append(dict(rec, us=round(ms * 1e3, 2)))
        print(f"# sample {i}: {recs[-1]}", file=sys.stderr, flush=True)
        pt.release()
    train = list(range(0, len(lat), 2))
    test = list(range(1, len(lat), 2))
    m = LatencyModel.fit([feats[i] for i in train], [lat[i] for i in train])
    held = m.residuals([feats[i] for i in test], [lat[i] for i in test])
    m_all = LatencyModel.fit(feats, lat)
    print(json.dumps({"latency_model": {
        "workload": f"{cfg.name} layer ({key}): random decode sets (8-256 decodes, contexts "
                    f"U[64, 4096]) with 0-4096-token chunks at prior context 0-4096",
        "coef_us": m.as_dict(), "held_out_residuals": held,
        "coef_us_all_samples": m_all.as_dict(),
        "in_sample_residuals_all": m_all.residuals(feats, lat), "samples": recs}}))


def main():
    args = parse()
    if args.summarize_stats:
        summarize_stats(*args.summarize_stats)
        return
    if args.summarize_traffic:
        a = args.summarize_traffic
        if len(a) not in (5, 7):
            sys.exit("--summarize-traffic takes 5 or 7 arguments")
        summarize_traffic(*a)
        return
    if args.simulate:
        from paper_2606_16264_amd.sched import LatencyModel, attainment_sweep
        import workload as wl
        rec = json.load(open(args.simulate))["latency_model"]
        cfg = wl.CONFIGS[args.config]
        noise = rec["held_out_residuals"]["median_abs_rel"]
        res = attainment_sweep(LatencyModel.from_dict(rec["coef_us"]), args.rates,
                               n=args.requests, kv_bytes_per_token=32.0 * cfg.kv_bytes_per_token,
                               noise=noise)
        res.update(latency_model=rec["workload"], noise=noise, layers=32,
                   workers="4 (2 prefill + 2 multiplexing)",
                   requests=args.requests,
                   arrivals="Poisson; prompts lognormal(median 2048, sigma 1) in [32, 16384]; "
                            "outputs lognormal(median 128, sigma 0.8) in [1, 1024]")
        print(json.dumps(res))
        return
    if args.predictor and args.predictor < 12:
        sys.exit("--predictor needs at least 12 batches: the model's six coefficients are fitted "
                 "on the even-numbered half")
    if args.gpus != 1:
        print(json.dumps({"error": "the layer step runs on one GPU; --gpus must be 1 "
                                   "(there is no multi-GPU path)"}))
        sys.exit(2)
    import numpy as np
    import torch
    import paper_2606_16264_amd as mx
    import workload as wl

    torch.cuda.set_device(0)
    key = args.config
    cfg = wl.CONFIGS[key]
    sweep = args.prefill if args.prefill is not None else wl.SWEEPS[key]
    w_host = wl.make_weights(cfg, key)
    w_dev = {k: torch.from_numpy(v).cuda() for k, v in w_host.items()}
    b0 = wl.make_batch(key, sweep[0])
    c0 = mx.layer_cfg(cfg.hidden, cfg.ffn, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                      b0.pool_pages, cfg.rms_eps, cfg.rope_theta)
    packed = torch.empty(mx.mx_packed_weights_bytes(c0), dtype=torch.uint8, device="cuda")
    mx.mx_pack_weights(c0, w_dev, packed)
    del w_dev
    torch.cuda.synchronize()
    if args.copy_calib_mib:
        n = args.copy_calib_mib << 20
        src = torch.ones(n, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"# copy calibration: {n} bytes device-to-device", file=sys.stderr, flush=True)
        del src, dst
    if args.chunk_sweep:
        chunk_sweep(args, key, cfg, packed)
        return
    if args.predictor:
        predictor_fit(args, key, cfg, packed)
        return
    print(f"# bench: {key} ({cfg.name}) sweep P={sweep}, steps={args.steps}, warmup={args.warmup}",
          file=sys.stderr, flush=True)

    curve = []
    headline = None
    kernels = {}
    for P in sweep:
        pt = Point(key, P, None, packed, cfg)
        torch.cuda.synchronize()
        ms, dist = time_fn(pt.step, args.steps, args.warmup)
        us = ms * 1e3
        roof = t_roof(pt.parts) * 1e6
        rec = dict(P=int(P), T=pt.b.T, R=pt.b.R, us=round(us, 2),
                   host_us=round(dist["host"] * 1e3, 1),
                   us_median=round(dist["median"] * 1e3, 2), us_p10=round(dist["p10"] * 1e3, 2),
                   us_p90=round(dist["p90"] * 1e3, 2),
                   tokens_per_s=pt.b.T / (us * 1e-6),
                   decode_tokens_per_s=int((pt.b.phase == wl.DECODE).sum()) / (us * 1e-6),
                   t_roof_us=round(roof, 2), roof_frac=roof / us)
        print(f"# P={P}: {us:.1f} us/step (median {rec['us_median']}, p10 {rec['us_p10']}, "
              f"p90 {rec['us_p90']}), {rec['tokens_per_s']:.0f} tok/s, "
              f"roofline {roof:.1f} us ({rec['roof_frac']:.2f}), host {rec['host_us']} us/step",
              file=sys.stderr, flush=True)
        if args.kernels:
            kernels = kernel_breakdown(pt, max(5, args.steps // 2), 2)
            rec["kernel_us"] = {k: round(v["us"], 2) for k, v in kernels.items()}
            pa = kernels.get("paged_attn")
            if pa:
                rec["attn_hbm_frac"] = round(pa["hbm_frac"], 4)
                rec["attn_mfma_frac"] = round(pa["mfma_frac"], 4)
            for k, v in kernels.items():
                print(f"#   kernel {k}: {v['us']:.1f} us  hbm_frac={v['hbm_frac']:.3f}  "
                      f"mfma_frac={v['mfma_frac']:.3f}", file=sys.stderr, flush=True)
        if P == sweep[-1]:
            headline = (pt, rec)
        else:
            pt.release()
        curve.append(rec)
    pt, rec = headline
    fit = linear_fit([c["P"] for c in curve], [c["us"] for c in curve])
    # dominant kernel and its roofline: the attention is HBM-bound (decode
    # K/V streaming), the projections MFMA-bound at these token counts
    dom = max(kernels, key=lambda k: kernels[k]["us"]) if kernels else None
    roofline = None
    wl_tag = f"{key}_P{pt.b.prefill_tokens}"
    if dom == "paged_attn":
        kv = kernels[dom]
        roofline = {"kernel": "paged_attn_kernel", "bound": "hbm",
                    "achieved": round(kv["achieved_GBps"], 1), "peak": HBM_PEAK / 1e9,
                    "unit": "GB/s", "frac": round(kv["hbm_frac"], 4),
                    "algorithmic_bytes": kv["bytes"], "avg_launch_us": round(kv["us"], 2),
                    "traffic": measured_traffic("paged_attn_kernel", wl_tag,
                                                "paper_2606_16264_amd/csrc/attention.hip")}
    elif dom is not None:
        kv = kernels[dom]
        roofline = {"kernel": dom, "bound": "mfma", "achieved": round(kv["TFLOPs"], 1),
                    "peak": MFMA_BF16_PEAK / 1e12, "unit": "TFLOP/s",
                    "frac": round(kv["mfma_frac"], 4), "algorithmic_flops": kv["flops"],
                    "avg_launch_us": round(kv["us"], 2),
                    "traffic": measured_traffic(dom, wl_tag, "paper_2606_16264_amd/csrc/gemm.hip")}
    cpu = None
    if not args.no_cpu:
        cpu = cpu_baseline(key, cfg, w_host, args.cpu_seconds)
    out = {
        "metric": METRIC,
        "value": round(rec["tokens_per_s"], 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(rec["us"] / 1e3, 5),
        "latency_us": rec["us"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (seeded; chat-style mixed batch shapes, random-init weights)",
        "config": {"workload": f"{cfg.name} layer ({key}): hidden {cfg.hidden}, "
                               f"{cfg.n_q_heads}q/{cfg.n_kv_heads}kv x {cfg.head_dim}, ffn {cfg.ffn}; "
                               f"{int((pt.b.phase == wl.DECODE).sum())} decodes + "
                               f"{pt.b.prefill_tokens} mixed prefill tokens",
                   "T": pt.b.T, "R": pt.b.R, "P": pt.b.prefill_tokens},
        "curve": curve,
        "curve_fit": fit,
        "t_roof_us": rec["t_roof_us"],
        "roof_frac": round(rec["roof_frac"], 4),
        "roofline": roofline,
        "kernels": {k: {m: (round(v, 4) if isinstance(v, float) else v) for m, v in d.items()}
                    for k, d in kernels.items()},
        "cpu_baseline": cpu,
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
