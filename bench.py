"""Benchmark of the QuantWM hot path on one MI355X.

One step = quantize-on-append of one chunk of new Key/Value tokens
(quantwm_append) + attention of the Query chunk over the packed cache
(quantwm_attend), on the 40-head LingBot-World-like workload: cache 21 frames x
1,560 tokens = 32,760 per head, Query chunk and append chunk 3 frames x 1,560 =
4,680 tokens, 128 centroids, group 32, r = 16, M = 4, bf16. Inputs are seeded
synthetic tensors (synth.py) resident in HBM before timing starts; the cache is
prefilled, and every step re-appends the last chunk into its slots (so each step
does identical work) and then attends.

Prints one JSON line. `value` is cache tokens/s of the whole step
(B * H * n_cache per step); the line also carries the per-kernel times, append
GB/s, the roofline of the dominant kernel (attend, bf16 matrix cores) measured
with HIP events on the launch stream, and the CPU oracle timed on a bounded
sample on this host.
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

import synth  # noqa: E402

PEAK_BF16_TFLOPS = 2516.6   # MI355X dense bf16 matrix peak
PEAK_FP32_VALU_TFLOPS = 78.6  # fp32 FMA on the vector ALUs without packed FP32
PEAK_HBM_GBPS = 8000.0


def visible_pairs(wl: synth.Workload) -> int:
    """Key-Query pairs the block-causal mask lets through, per (b, h)."""
    i = np.arange(wl.n_q)
    lim = np.minimum(wl.n_cache, wl.q_start + (i // wl.frame_tokens + 1) * wl.frame_tokens)
    return int(lim.sum())


def attend_flops(wl) -> float:
    bh = wl.batch * wl.heads
    return bh * (visible_pairs(wl) * (4 * wl.head_dim + 2 * wl.rank) + 2 * wl.n_q * wl.head_dim * wl.rank)


def token_bytes(wl):
    ng = wl.head_dim // wl.group_size
    v = wl.head_dim // 4 + 1 + (ng + 3) // 4 + 2 * ng
    return v + (wl.rank + 2 if wl.rank else 0), v


def append_bytes(wl, n_new) -> float:
    kb, vb = token_bytes(wl)
    e = 2 if wl.dtype == "bf16" else 4
    return wl.batch * wl.heads * n_new * (2 * wl.head_dim * e + kb + vb)


def append_flops(wl, n_new) -> float:
    d = wl.head_dim
    return wl.batch * wl.heads * n_new * (4 * wl.n_centroids * d + 2 * d * wl.rank + 28 * d)


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter summary of this
    workload, or None when there is none or the kernel source has changed since
    the counters were taken (the summary records the source's SHA-256)."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"attend_append_{workload}_traffic.md")
    src = os.path.join(ROOT, "paper_2609_26425_amd", "csrc", f"{kernel}.hip")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.split(":")[0].strip().startswith(kernel + "_"):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    digest = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if fields.get(f"{kernel}_source_sha256") != digest or f"{kernel}_traffic_bytes_per_launch" not in fields:
        return None
    return int(fields[f"{kernel}_traffic_bytes_per_launch"])


def cpu_baseline(wl):
    """The oracle as it stands, timed on a bounded sample of the same step."""
    import oracle
    if not os.path.exists(oracle.LIB):
        oracle.build()
    threads = oracle.max_threads()
    nh = max(1, min(threads, wl.batch * wl.heads))
    heads = [divmod(i, wl.heads) for i in range(nh)]
    cfg = oracle.cfg_of(1, nh, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m, wl.n_cache,
                        wl.dtype == "bf16")

    def gen(fn, n):
        out = np.zeros((1, n, nh, wl.head_dim), np.float32)
        for s, (b, h) in enumerate(heads):
            out[0, :, s, :] = synth.round_to(fn(wl, b, h, n), wl.dtype)
        return out

    k = gen(synth.keys_head, wl.chunk)
    v = gen(synth.values_head, wl.chunk)
    qh = gen(lambda w, b, h, n: synth.queries_head(w, b, h, n, True), wl.n_hist)
    tables = oracle.calibrate(cfg, qh, k, v, wl.kmeans_iters)
    # append leg: one chunk on nh heads in parallel, scaled to every head
    cache = oracle.new_cache(cfg)
    t0 = time.perf_counter()
    oracle.append(cfg, tables, cache, wl.n_cache - wl.chunk, k, v)
    t_app = (time.perf_counter() - t0) * (wl.batch * wl.heads) / nh
    # attend leg: head 0 with a full cache, every 16th Query row, scaled by visible pairs
    cfg1 = oracle.cfg_of(1, 1, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m, wl.n_cache,
                         wl.dtype == "bf16")
    t1 = tuple(np.ascontiguousarray(t[:, :1]) for t in tables)
    kf = synth.round_to(synth.keys_head(wl, 0, 0, wl.n_cache), wl.dtype)[None, :, None, :]
    vf = synth.round_to(synth.values_head(wl, 0, 0, wl.n_cache), wl.dtype)[None, :, None, :]
    q = synth.round_to(synth.queries_head(wl, 0, 0, wl.n_q), wl.dtype)[None, :, None, :]
    cache1 = oracle.new_cache(cfg1)
    oracle.append(cfg1, t1, cache1, 0, kf, vf)
    rows = np.array([(0, 0, i) for i in range(0, wl.n_q, 16)], np.int32)
    t0 = time.perf_counter()
    oracle.attend(cfg1, t1, cache1, wl.n_cache, q, wl.q_start, wl.frame_tokens, rows=rows)
    t_sample = time.perf_counter() - t0
    i = rows[:, 2]
    lim = np.minimum(wl.n_cache, wl.q_start + (i // wl.frame_tokens + 1) * wl.frame_tokens)
    t_att = t_sample * (visible_pairs(wl) / float(lim.sum())) * wl.batch * wl.heads
    t_step = t_app + t_att
    # the same legs on one thread: one head's append, every 64th Query row
    oracle.set_threads(1)
    try:
        c1 = oracle.cfg_of(1, 1, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m, wl.n_cache,
                           wl.dtype == "bf16")
        cache_s = oracle.new_cache(c1)
        t0 = time.perf_counter()
        oracle.append(c1, t1, cache_s, wl.n_cache - wl.chunk, np.ascontiguousarray(k[:, :, :1]),
                      np.ascontiguousarray(v[:, :, :1]))
        t_app1 = (time.perf_counter() - t0) * wl.batch * wl.heads
        rows1 = rows[::4]
        t0 = time.perf_counter()
        oracle.attend(cfg1, t1, cache1, wl.n_cache, q, wl.q_start, wl.frame_tokens, rows=rows1)
        t_s1 = time.perf_counter() - t0
        i1 = rows1[:, 2]
        lim1 = np.minimum(wl.n_cache, wl.q_start + (i1 // wl.frame_tokens + 1) * wl.frame_tokens)
        t_att1 = t_s1 * (visible_pairs(wl) / float(lim1.sum())) * wl.batch * wl.heads
    finally:
        oracle.set_threads(threads)
    single = {"value": wl.batch * wl.heads * wl.n_cache / (t_app1 + t_att1), "cores": 1,
              "sample": f"append of one head's {wl.chunk}-token chunk; attend of {len(rows1)} Query rows of one head",
              "append_s_est": t_app1, "attend_s_est": t_att1}
    cpu_model = None
    try:
        with open("/proc/cpuinfo") as f:
            cpu_model = next((ln.split(":", 1)[1].strip() for ln in f if ln.startswith("model name")), None)
    except OSError:
        pass
    return {"value": wl.batch * wl.heads * wl.n_cache / t_step, "unit": "cache tokens/s", "cores": threads,
            "cpu_model": cpu_model, "host_cpus": os.cpu_count(),
            "kind": "oracle",
            "sample": (f"append of one {wl.chunk}-token chunk on {nh} heads (one OpenMP thread per head), "
                       f"scaled to {wl.batch * wl.heads} heads; attend of {len(rows)} of {wl.n_q} Query rows of "
                       f"one head over {wl.n_cache} keys ({threads} threads over rows), scaled by visible pairs "
                       f"to all rows and heads"),
            "append_s_est": t_app, "attend_s_est": t_att, "single_thread": single}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="lingbot-40h", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--copies", type=int, default=3, help="rotated input/cache copies (defeats the 256 MiB MALL)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-streaming", action="store_true",
                    help="skip the active-chunk and calibration-epoch timings (for kernel traces)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="also run one plain 1 GiB device copy kernel (read 1 GiB, write 1 GiB) outside the timed "
                         "region, as the scale for FETCH_SIZE / WRITE_SIZE counter runs")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the library has no multi-GPU path (heads would shard across GPUs "
              "with no exchange). Run with --gpus 1.", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_26425_amd import quantwm as qw

    wl = synth.WORKLOADS[args.workload]
    dev = "cuda:0"
    torch.cuda.set_device(0)
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    cfg = qw.make_config(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m,
                         wl.n_cache, wl.dtype)
    print(f"[bench] generating {wl.name} inputs", file=sys.stderr, flush=True)
    k_all = torch.from_numpy(synth.tensor(wl, "k", wl.n_cache)).to(dev, dt)
    v_all = torch.from_numpy(synth.tensor(wl, "v", wl.n_cache)).to(dev, dt)
    qh = torch.from_numpy(synth.tensor(wl, "qhist", wl.n_hist)).to(dev, dt)
    q = torch.from_numpy(synth.tensor(wl, "q", wl.n_q)).to(dev, dt)

    print("[bench] calibrating", file=sys.stderr, flush=True)
    calib = torch.zeros(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=dev)
    ws = torch.empty(qw.quantwm_calibrate_workspace_bytes(cfg, wl.n_hist, wl.chunk), dtype=torch.uint8, device=dev)
    qw.quantwm_calibrate(cfg, qh, wl.n_hist, k_all[:, :wl.chunk].contiguous(), v_all[:, :wl.chunk].contiguous(),
                         wl.chunk, wl.kmeans_iters, calib, ws)
    del ws

    n_new = wl.chunk
    start = wl.n_cache - n_new
    caches, k_new, v_new = [], [], []
    print("[bench] prefilling caches", file=sys.stderr, flush=True)
    for c in range(args.copies):
        cache = torch.zeros(qw.quantwm_cache_bytes(cfg), dtype=torch.uint8, device=dev)
        for s0, n in wl.chunks():
            qw.quantwm_append(cfg, calib, cache, s0, k_all[:, s0:s0 + n].contiguous(),
                              v_all[:, s0:s0 + n].contiguous(), n)
        caches.append(cache)
        k_new.append(k_all[:, start:].contiguous().clone())
        v_new.append(v_all[:, start:].contiguous().clone())
    outs = [torch.empty_like(q) for _ in range(args.copies)]
    qs = [q.clone() for _ in range(args.copies)]
    lse = torch.empty((wl.batch, wl.heads, wl.n_q), dtype=torch.float32, device=dev)
    ws_bytes = qw.quantwm_attend_workspace_bytes(cfg, wl.n_cache, wl.n_q)
    attend_ws = torch.empty(ws_bytes, dtype=torch.uint8, device=dev) if ws_bytes else None
    del k_all, v_all
    torch.cuda.synchronize()

    def step(i, ev=None):
        c = i % args.copies
        if ev is not None:
            ev[0].record()
        qw.quantwm_append(cfg, calib, caches[c], start, k_new[c], v_new[c], n_new)
        if ev is not None:
            ev[1].record()
        qw.quantwm_attend(cfg, calib, caches[c], wl.n_cache, qs[c], wl.n_q, wl.q_start, wl.frame_tokens,
                          outs[c], lse, attend_ws)
        if ev is not None:
            ev[2].record()

    if args.copy_probe:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)  # elementwise kernel: 1 GiB read, 1 GiB written
        torch.cuda.synchronize()
        del src, dst

    print(f"[bench] warmup {args.warmup}", file=sys.stderr, flush=True)
    for i in range(args.warmup):
        step(i)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    print(f"[bench] timing {args.steps} steps", file=sys.stderr, flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i, evs[i])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    app_all = np.array([e[0].elapsed_time(e[1]) for e in evs])
    att_all = np.array([e[1].elapsed_time(e[2]) for e in evs])
    app_ms, att_ms = float(app_all.mean()), float(att_all.mean())
    ms_step = wall * 1000.0 / args.steps
    assert torch.isfinite(outs[0].float()).all(), "non-finite attention output"

    # the streaming forms, timed separately on the same inputs (skipped with
    # --no-streaming, so that a kernel trace holds the step's launches only: the
    # per-epoch and two-part forms launch the same plain attention kernel)
    act_ms = ep_ms = act_cfg = ep_cfg = None
    if not args.no_streaming:
        # the streaming variant: the last chunk stays exact (BF16) beside the packed
        # history of the rest, timed separately on the same inputs
        n_pk = wl.n_cache - n_new
        ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        # with the two-part workspace: packed whole tiles through the plain kernel,
        # the rest through the general one, merged by log-sum-exp
        ws_act = qw.quantwm_attend_active_workspace_bytes(cfg, n_pk, n_new, wl.n_q)
        act_ws = torch.empty(ws_act, dtype=torch.uint8, device=dev) if ws_act else None
        for i in range(2):
            qw.quantwm_attend_active(cfg, calib, caches[0], n_pk, k_new[0], v_new[0], n_new, qs[0], wl.n_q,
                                     wl.q_start, wl.frame_tokens, outs[0], lse, act_ws)
        ea.record()
        for i in range(5):
            qw.quantwm_attend_active(cfg, calib, caches[0], n_pk, k_new[0], v_new[0], n_new, qs[0], wl.n_q,
                                     wl.q_start, wl.frame_tokens, outs[0], lse, act_ws)
        eb.record()
        torch.cuda.synchronize()
        act_ms = ea.elapsed_time(eb) / 5

        # calibration epochs: one per appended chunk (the timing does not depend on
        # the tables' values, so every epoch reuses this calibration block)
        starts = [s0 for s0, _ in wl.chunks()]
        cb = qw.quantwm_calib_bytes(cfg)
        calibs = calib.repeat(len(starts))
        # with the per-epoch workspace: each epoch's keys through the plain kernel,
        # merged by log-sum-exp
        ws_ep = qw.quantwm_attend_epochs_workspace_bytes(cfg, starts, wl.n_cache, 0, wl.n_q)
        ep_ws = torch.empty(ws_ep, dtype=torch.uint8, device=dev) if ws_ep else attend_ws
        for i in range(2):
            qw.quantwm_attend_epochs(cfg, calibs, starts, caches[0], wl.n_cache, None, None, 0, qs[0], wl.n_q,
                                     wl.q_start, wl.frame_tokens, outs[0], lse, ep_ws)
        ea.record()
        for i in range(5):
            qw.quantwm_attend_epochs(cfg, calibs, starts, caches[0], wl.n_cache, None, None, 0, qs[0], wl.n_q,
                                     wl.q_start, wl.frame_tokens, outs[0], lse, ep_ws)
        eb.record()
        torch.cuda.synchronize()
        ep_ms = ea.elapsed_time(eb) / 5
        del calibs, cb, ep_ws
        act_cfg = f"{n_pk} packed + {n_new} exact BF16 keys, two-part workspace {ws_act} B"
        ep_cfg = f"{len(starts)} calibration epochs, one per {wl.chunk}-token chunk, per-epoch workspace {ws_ep} B"

    flops = attend_flops(wl)
    achieved = flops / (att_ms * 1e-3) / 1e12
    app_bytes = append_bytes(wl, n_new)
    app_gbps = app_bytes / (app_ms * 1e-3) / 1e9
    app_tflops = append_flops(wl, n_new) / (app_ms * 1e-3) / 1e12
    bh = wl.batch * wl.heads
    line = {
        "metric": "cache tokens/s for quantwm_attend + append GB/s (fraction of MI355X roofline)",
        "value": bh * wl.n_cache / (ms_step * 1e-3),
        "unit": "cache tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": f"{wl.name}: B={wl.batch} H={wl.heads} d={wl.head_dim} n_cache={wl.n_cache} "
                               f"n_q={wl.n_q} append={n_new} Kc={wl.n_centroids} G={wl.group_size} r={wl.rank} "
                               f"M={wl.top_m} F={wl.frame_tokens}",
                   "global_batch": wl.batch, "seq_len": wl.n_cache, "parallelism": "single GPU"},
        "attend_ms": att_ms, "append_ms": app_ms,
        "attend_ms_median_min": [float(np.median(att_all)), float(att_all.min())],
        "append_ms_median_min": [float(np.median(app_all)), float(app_all.min())],
        "attend_cache_tokens_per_s": bh * wl.n_cache / (att_ms * 1e-3),
        "append_GBps": app_gbps,
        "append_hbm_frac": app_gbps / PEAK_HBM_GBPS,
        "append_valu_frac": app_tflops / PEAK_FP32_VALU_TFLOPS,
        "roofline": {"kernel": "attend", "bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": achieved / PEAK_BF16_TFLOPS,
                     "traffic": measured_traffic("attend", wl.name)},
        "append_traffic": measured_traffic("append", wl.name),
        "copies": args.copies,
        "attend_workspace_bytes": ws_bytes,
        "attend_active_ms": act_ms,
        "attend_active_config": act_cfg,
        "attend_epochs_ms": ep_ms,
        "attend_epochs_config": ep_cfg,
    }
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
