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
with HIP events on the launch stream, the streaming forms (active chunk,
calibration epochs), one record per other configuration under "workloads"
(tiny fp32, Matrix-Game-like, batched, and the long rollout at 30k, 60k and
120k cached tokens: the same step, timed the same way, on 4 synthetic source
heads repeated over the launch), and the CPU oracle timed on a bounded sample
on this host.
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
PEAK_FP32_MFMA_TFLOPS = 157.3  # fp32 matrix peak (the tiny fp32 workload)


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
    """Algorithmic flops of one append call: the two centroid searches (2 Kc d
    each), PSAC (2 d r) and about 28 per channel for the Eq. 12 score and the
    residuals."""
    d = wl.head_dim
    return wl.batch * wl.heads * n_new * (4 * wl.n_centroids * d + 2 * d * wl.rank + 28 * d)


# the device-code sources of each kernel (their digest dates a counter summary)
KERNEL_SOURCES = {"attend": ["attend.hip", "attend_host.hip", "attend_shape.h", "qwm_common.h", "xcd_order.h"],
                  "append": ["append_bf16.hip", "append.hip", "append_common.h", "qwm_common.h", "xcd_order.h"]}


def source_digest(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        h.update(open(os.path.join(ROOT, "paper_2609_26425_amd", "csrc", f), "rb").read())
    return h.hexdigest()


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch of `kernel` from the committed counter summary of this
    workload, or None when there is none or the kernel sources have changed
    since the counters were taken (the summary records their SHA-256)."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and line.split(":")[0].strip().startswith(kernel + "_"):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    if fields.get(f"{kernel}_source_sha256") != source_digest(kernel) or \
            f"{kernel}_traffic_bytes_per_launch" not in fields:
        return None
    return int(fields[f"{kernel}_traffic_bytes_per_launch"])


def attend_bytes(wl) -> float:
    """Algorithmic HBM bytes of one attention launch: the packed cache read once,
    the Queries read, the outputs and lse written."""
    kb, vb = token_bytes(wl)
    e = 2 if wl.dtype == "bf16" else 4
    bh = wl.batch * wl.heads
    return bh * (wl.n_cache * (kb + vb) + wl.n_q * wl.head_dim * 2 * e + wl.n_q * 4)


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


def replicated_inputs(wl, what, n, sources):
    """[B, n, H, d] float32 where head (b, h) carries synthetic head sources[(b H + h)
    % S]: the generator's own heads, S of them, repeated over the launch (the
    timing does not depend on which head's values a head holds)."""
    fn = {"k": synth.keys_head, "v": synth.values_head,
          "q": lambda w, b, h, m: synth.queries_head(w, b, h, m, False),
          "qhist": lambda w, b, h, m: synth.queries_head(w, b, h, m, True)}[what]
    src = [synth.round_to(fn(wl, b, h, n), wl.dtype) for (b, h) in sources]
    out = np.empty((wl.batch, n, wl.heads, wl.head_dim), np.float32)
    for bh in range(wl.batch * wl.heads):
        b, h = divmod(bh, wl.heads)
        out[b, :, h, :] = src[bh % len(sources)]
    return out


class Prepared:
    """A workload's calibration block, rotated caches (prefilled by append) and
    inputs, resident on the GPU."""

    def __init__(self, wl, copies, n_sources=None):
        import torch
        from paper_2609_26425_amd import quantwm as qw
        self.wl, self.qw, self.copies = wl, qw, copies
        dev = "cuda:0"
        dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
        self.cfg = cfg = qw.make_config(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank,
                                        wl.top_m, wl.n_cache, wl.dtype)
        if n_sources is None:
            gen = lambda what, n: synth.tensor(wl, what, n)  # noqa: E731
        else:
            allh = [(b, h) for b in range(wl.batch) for h in range(wl.heads)]
            srcs = allh[:n_sources]
            gen = lambda what, n: replicated_inputs(wl, what, n, srcs)  # noqa: E731
        k_all = torch.from_numpy(gen("k", wl.n_cache)).to(dev, dt)
        v_all = torch.from_numpy(gen("v", wl.n_cache)).to(dev, dt)
        qh = torch.from_numpy(gen("qhist", wl.n_hist)).to(dev, dt)
        q = torch.from_numpy(gen("q", wl.n_q)).to(dev, dt)
        self.calib = torch.zeros(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=dev)
        nc = min(wl.chunk, wl.n_cache)
        ws = torch.empty(qw.quantwm_calibrate_workspace_bytes(cfg, wl.n_hist, nc), dtype=torch.uint8, device=dev)
        qw.quantwm_calibrate(cfg, qh, wl.n_hist, k_all[:, :nc].contiguous(), v_all[:, :nc].contiguous(), nc,
                             wl.kmeans_iters, self.calib, ws)
        del ws
        self.n_new = n_new = nc
        self.start = wl.n_cache - n_new
        self.caches, self.k_new, self.v_new = [], [], []
        for c in range(copies):
            cache = torch.zeros(qw.quantwm_cache_bytes(cfg), dtype=torch.uint8, device=dev)
            for s0, n in wl.chunks():
                qw.quantwm_append(cfg, self.calib, cache, s0, k_all[:, s0:s0 + n].contiguous(),
                                  v_all[:, s0:s0 + n].contiguous(), n)
            self.caches.append(cache)
            self.k_new.append(k_all[:, self.start:].contiguous().clone())
            self.v_new.append(v_all[:, self.start:].contiguous().clone())
        self.outs = [torch.empty_like(q) for _ in range(copies)]
        self.qs = [q.clone() for _ in range(copies)]
        self.lse = torch.empty((wl.batch, wl.heads, wl.n_q), dtype=torch.float32, device=dev)
        self.ws_bytes = qw.quantwm_attend_workspace_bytes(cfg, wl.n_cache, wl.n_q)
        self.attend_ws = torch.empty(self.ws_bytes, dtype=torch.uint8, device=dev) if self.ws_bytes else None
        del k_all, v_all
        torch.cuda.synchronize()

    def step(self, i, ev=None):
        wl, qw, c = self.wl, self.qw, i % self.copies
        if ev is not None:
            ev[0].record()
        qw.quantwm_append(self.cfg, self.calib, self.caches[c], self.start, self.k_new[c], self.v_new[c], self.n_new)
        if ev is not None:
            ev[1].record()
        qw.quantwm_attend(self.cfg, self.calib, self.caches[c], wl.n_cache, self.qs[c], wl.n_q, wl.q_start,
                          wl.frame_tokens, self.outs[c], self.lse, self.attend_ws)
        if ev is not None:
            ev[2].record()

    def time(self, steps, warmup):
        """(wall seconds of `steps` steps, append ms per step, attend ms per step),
        the kernel times from HIP events on the launch stream."""
        import torch
        for i in range(warmup):
            self.step(i)
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for i in range(steps):
            self.step(i, evs[i])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        app = np.array([e[0].elapsed_time(e[1]) for e in evs])
        att = np.array([e[1].elapsed_time(e[2]) for e in evs])
        assert torch.isfinite(self.outs[0].float()).all(), "non-finite attention output"
        return wall, app, att


def kernel_record(wl, n_new, app_all, att_all, ws_bytes):
    """Per-kernel figures of one workload: times, rates and roofline fractions.
    ws_bytes: the attention workspace the launch took (its key-split planes)."""
    app_ms, att_ms = float(app_all.mean()), float(att_all.mean())
    bh = wl.batch * wl.heads
    splits = max(1, round(ws_bytes / (bh * wl.n_q * (4 * wl.head_dim + 8)))) if ws_bytes else 1
    fl = attend_flops(wl) / (att_ms * 1e-3) / 1e12
    ab = attend_bytes(wl)
    rec = {
        "attend_ms": att_ms, "attend_ms_median_min": [float(np.median(att_all)), float(att_all.min())],
        "append_ms": app_ms, "append_ms_median_min": [float(np.median(app_all)), float(app_all.min())],
        "attend_cache_tokens_per_s": bh * wl.n_cache / (att_ms * 1e-3),
        "attend_TFLOPs": fl, "attend_mfma_frac": fl / (PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_MFMA_TFLOPS),
        "attend_algorithmic_bytes": ab, "attend_GBps": ab / (att_ms * 1e-3) / 1e9,
        "attend_key_splits": splits,
        "append_tokens": bh * n_new,
        "append_GBps": append_bytes(wl, n_new) / (app_ms * 1e-3) / 1e9,
        # BF16 Keys and Values: the searches run on the matrix cores and the rest
        # (selection, Eq. 12 score, residuals, PSAC) on the vector ALU, so no
        # single peak bounds the kernel; fp32 ones run everything on the vector ALU
        "append_search_on": "mfma" if wl.dtype == "bf16" else "valu",
        "append_algorithmic_TFLOPs": append_flops(wl, n_new) / (app_ms * 1e-3) / 1e12,
    }
    if wl.dtype != "bf16":
        rec["append_valu_frac"] = append_flops(wl, n_new) / (app_ms * 1e-3) / 1e12 / PEAK_FP32_VALU_TFLOPS
    rec["append_hbm_frac"] = rec["append_GBps"] / PEAK_HBM_GBPS
    for k in ("attend", "append"):
        t = measured_traffic(k, wl.name)
        rec[f"{k}_traffic_bytes"] = t
        if t is not None:
            rec[f"{k}_traffic_GBps"] = t / ((att_ms if k == "attend" else app_ms) * 1e-3) / 1e9
    return rec


def workload_desc(wl, n_new):
    return (f"{wl.name}: B={wl.batch} H={wl.heads} d={wl.head_dim} n_cache={wl.n_cache} n_q={wl.n_q} "
            f"append={n_new} Kc={wl.n_centroids} G={wl.group_size} r={wl.rank} M={wl.top_m} F={wl.frame_tokens}")


SUB_WORKLOADS = ["tiny-f32", "mg2-12h", "batched-4x30h", "rollout-30k", "rollout-60k", "rollout-120k"]


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
    ap.add_argument("--no-sub", action="store_true",
                    help="skip the per-workload records of the other configurations (for kernel traces)")
    ap.add_argument("--sub-steps", type=int, default=10)
    ap.add_argument("--sources", type=int, default=0,
                    help="generate this many synthetic heads and repeat them over the launch (0: every head)")
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
    print(f"[bench] {wl.name}: inputs, calibration, prefill of {args.copies} caches", file=sys.stderr, flush=True)
    P = Prepared(wl, args.copies, n_sources=args.sources or None)
    cfg, calib, n_new = P.cfg, P.calib, P.n_new

    if args.copy_probe:
        src = torch.ones(1 << 28, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.mul(src, 1.0, out=dst)  # elementwise kernel: 1 GiB read, 1 GiB written
        torch.cuda.synchronize()
        del src, dst

    print(f"[bench] warmup {args.warmup}, timing {args.steps} steps", file=sys.stderr, flush=True)
    wall, app_all, att_all = P.time(args.steps, args.warmup)
    app_ms, att_ms = float(app_all.mean()), float(att_all.mean())
    ms_step = wall * 1000.0 / args.steps

    # the streaming forms, timed separately on the same inputs (skipped with
    # --no-streaming, so that a kernel trace holds the step's launches only: the
    # per-epoch and two-part forms launch the same plain attention kernel)
    act_ms = ep_ms = act_cfg = ep_cfg = None
    if not args.no_streaming:
        # the last chunk stays exact (BF16) beside the packed history of the rest;
        # with the two-part workspace: packed whole tiles through the plain kernel,
        # the rest through the general one, merged by log-sum-exp
        n_pk = wl.n_cache - n_new
        ea, eb = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ws_act = qw.quantwm_attend_active_workspace_bytes(cfg, n_pk, n_new, wl.n_q)
        act_ws = torch.empty(ws_act, dtype=torch.uint8, device=dev) if ws_act else None

        def active():
            qw.quantwm_attend_active(cfg, calib, P.caches[0], n_pk, P.k_new[0], P.v_new[0], n_new, P.qs[0], wl.n_q,
                                     wl.q_start, wl.frame_tokens, P.outs[0], P.lse, act_ws)
        for i in range(2):
            active()
        ea.record()
        for i in range(5):
            active()
        eb.record()
        torch.cuda.synchronize()
        act_ms = ea.elapsed_time(eb) / 5

        # calibration epochs: one per appended chunk (the timing does not depend on
        # the tables' values, so every epoch reuses this calibration block); with
        # the per-epoch workspace each epoch's keys go through the plain kernel
        starts = [s0 for s0, _ in wl.chunks()]
        calibs = calib.repeat(len(starts))
        ws_ep = qw.quantwm_attend_epochs_workspace_bytes(cfg, starts, wl.n_cache, 0, wl.n_q)
        ep_ws = torch.empty(ws_ep, dtype=torch.uint8, device=dev) if ws_ep else P.attend_ws

        def epochs():
            qw.quantwm_attend_epochs(cfg, calibs, starts, P.caches[0], wl.n_cache, None, None, 0, P.qs[0], wl.n_q,
                                     wl.q_start, wl.frame_tokens, P.outs[0], P.lse, ep_ws)
        for i in range(2):
            epochs()
        ea.record()
        for i in range(5):
            epochs()
        eb.record()
        torch.cuda.synchronize()
        ep_ms = ea.elapsed_time(eb) / 5
        del calibs, ep_ws, act_ws
        act_cfg = f"{n_pk} packed + {n_new} exact BF16 keys, two-part workspace {ws_act} B"
        ep_cfg = f"{len(starts)} calibration epochs, one per {wl.chunk}-token chunk, per-epoch workspace {ws_ep} B"

    rec = kernel_record(wl, n_new, app_all, att_all, P.ws_bytes)
    bh = wl.batch * wl.heads
    line = {
        "metric": "cache tokens/s for quantwm_attend + append GB/s (fraction of MI355X roofline)",
        "value": bh * wl.n_cache / (ms_step * 1e-3),
        "unit": "cache tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": wl.dtype, "data": "synthetic",
        "config": {"workload": workload_desc(wl, n_new),
                   "global_batch": wl.batch, "seq_len": wl.n_cache, "parallelism": "single GPU"},
        "attend_ms": att_ms, "append_ms": app_ms,
        "attend_ms_median_min": rec["attend_ms_median_min"],
        "append_ms_median_min": rec["append_ms_median_min"],
        "attend_cache_tokens_per_s": rec["attend_cache_tokens_per_s"],
        "attend_GBps": rec["attend_GBps"],
        "attend_key_splits": rec["attend_key_splits"],
        "append_GBps": rec["append_GBps"],
        "append_hbm_frac": rec["append_hbm_frac"],
        "append_search_on": rec["append_search_on"],
        "append_algorithmic_TFLOPs": rec["append_algorithmic_TFLOPs"],
        "roofline": {"kernel": "attend", "bound": "mfma", "achieved": rec["attend_TFLOPs"], "peak": PEAK_BF16_TFLOPS,
                     "unit": "TFLOP/s", "frac": rec["attend_TFLOPs"] / PEAK_BF16_TFLOPS,
                     "traffic": rec["attend_traffic_bytes"]},
        "append_traffic": rec["append_traffic_bytes"],
        "copies": args.copies,
        "attend_workspace_bytes": P.ws_bytes,
        "attend_active_ms": act_ms,
        "attend_active_config": act_cfg,
        "attend_epochs_ms": ep_ms,
        "attend_epochs_config": ep_cfg,
    }
    del P
    torch.cuda.empty_cache()

    # every other configuration: one append + one attend per step, as the
    # headline, on 4 synthetic source heads repeated over the launch
    if not args.no_sub:
        subs = {}
        for name in SUB_WORKLOADS:
            if name == wl.name:
                continue
            w = synth.WORKLOADS[name]
            print(f"[bench] sub-record {name}", file=sys.stderr, flush=True)
            S = Prepared(w, args.copies, n_sources=4)
            _, a_all, t_all = S.time(args.sub_steps, 3)
            r = kernel_record(w, S.n_new, a_all, t_all, S.ws_bytes)
            r["config"] = workload_desc(w, S.n_new)
            r["attend_workspace_bytes"] = S.ws_bytes
            r["data"] = "synthetic, 4 source heads repeated over the launch"
            subs[name] = r
            del S
            torch.cuda.empty_cache()
        line["workloads"] = subs
    if not args.no_cpu_baseline:
        print("[bench] timing the CPU oracle on a sample", file=sys.stderr, flush=True)
        line["cpu_baseline"] = cpu_baseline(wl)
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
