"""Synthetic quality harness for the packed cache.

For a seeded synthetic workload this measures how far the attention logits over
the packed cache move from the exact ones, for the four settings the paper
ablates (Sec. 5, the component ablation): plain nearest-centroid quantisation
(M = 1, w = 1, r = 0, the QVG setting), QSAC alone (r = 0), PSAC alone (M = 1,
w = 1) and both; a sweep over the candidate count M; both with the App. D.1
storage options; and both with the candidates ranked by the full quadratic form
of the Query second moment instead of its diagonal (App. C). The metrics are
taken over the visible (Query, key) pairs of the first `n_eval` Queries of the
chunk:

* logit MSE, and the RMS logit error relative to the RMS of the exact logits;
* the top-1 token-shift ratio: the share of Queries whose highest-logit key
  changes (Sec. 3, the token-shift analysis).

Every quantised logit comes from the library (quantwm_append and the
quantwm_logits hook); the exact ones are fp32 products of the same BF16 inputs.
Prints one JSON object.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

# mode -> (top_m or None for the workload's M, w forced to 1, PSAC on)
MODES = {
    "qvg": (1, True, False),
    "qsac": (None, False, False),
    "psac": (1, True, True),
    "both": (None, False, True),
}


def visible_mask(wl, n_eval: int, n_keys: int) -> np.ndarray:
    """[n_eval, n_keys] block-causal visibility (Query i at position q_start + i)."""
    i = np.arange(n_eval)[:, None]
    j = np.arange(n_keys)[None, :]
    return (j < wl.q_start) | ((j - wl.q_start) // wl.frame_tokens <= i // wl.frame_tokens)


def metrics(exact: np.ndarray, quant: np.ndarray, visible: np.ndarray) -> dict:
    """exact, quant: [..., n_eval, n_keys] logits; visible: [n_eval, n_keys]."""
    vis = np.broadcast_to(visible, exact.shape)
    diff = (quant.astype(np.float64) - exact.astype(np.float64))[vis]
    ex = exact.astype(np.float64)[vis]
    mse = float(np.mean(diff * diff))
    rel = math.sqrt(mse) / math.sqrt(float(np.mean(ex * ex)))
    e = np.where(vis, exact, -np.inf)
    q = np.where(vis, quant, -np.inf)
    shift = float(np.mean(np.argmax(e, axis=-1) != np.argmax(q, axis=-1)))
    return {"logit_mse": mse, "logit_rel_rms": rel, "top1_shift": shift}


def _torch():
    import torch
    from paper_2609_26425_amd import quantwm as qw
    return torch, qw


def gpu_tables(wl):
    """Calibrate on the GPU at the workload's (M, r) and read the tables back:
    (mu_k, mu_v, w, u_t, lam, m) as numpy arrays [B, H, ...]; m [B, H, d, d] is
    the full metric's matrix."""
    torch, qw = _torch()
    dev = "cuda:0"
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    cfg = qw.make_config(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m,
                         wl.n_cache, wl.dtype, metric=qw.METRIC_FULL)
    nc = min(wl.chunk, wl.n_cache)
    k = torch.from_numpy(synth.tensor(wl, "k", nc)).to(dev, dt)
    v = torch.from_numpy(synth.tensor(wl, "v", nc)).to(dev, dt)
    qh = torch.from_numpy(synth.tensor(wl, "qhist", wl.n_hist)).to(dev, dt)
    calib = torch.zeros(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=dev)
    ws = torch.empty(qw.quantwm_calibrate_workspace_bytes(cfg, wl.n_hist, nc), dtype=torch.uint8, device=dev)
    qw.quantwm_calibrate(cfg, qh, wl.n_hist, k, v, nc, wl.kmeans_iters, calib, ws)
    torch.cuda.synchronize()
    L = qw.quantwm_calib_offsets(cfg)
    BH, d, K, r = wl.batch * wl.heads, wl.head_dim, wl.n_centroids, wl.rank
    slabs = calib.view(BH, L.slab_bytes)

    def field(off, count, t):
        size = torch.tensor([], dtype=t).element_size()
        return slabs[:, off:off + count * size].contiguous().view(t).float().cpu().numpy()

    mu_k = field(L.mu_k, K * d, dt).reshape(wl.batch, wl.heads, K, d)
    mu_v = field(L.mu_v, K * d, dt).reshape(wl.batch, wl.heads, K, d)
    w = field(L.w, d, torch.float32).reshape(wl.batch, wl.heads, d)
    u_t = field(L.u_t, r * d, dt).reshape(wl.batch, wl.heads, r, d) if r else None
    lam = field(L.lam, r, torch.float32).reshape(wl.batch, wl.heads, r) if r else None
    m = field(L.m, d * d, torch.float32).reshape(wl.batch, wl.heads, d, d)
    return mu_k, mu_v, w, u_t, lam, m


def mode_tables(tables, wl, mode):
    """(config overrides, tables) of one mode from the calibrated tables; a sixth
    table (the full metric's matrix) is passed through."""
    top_m, w_one, psac = MODES[mode] if isinstance(mode, str) else mode
    mu_k, mu_v, w, u_t, lam = tables[:5]
    rank = wl.rank if psac else 0
    w_m = np.ones_like(w) if w_one else w
    return (top_m or wl.top_m, rank), (mu_k, mu_v, w_m, u_t if rank else None, lam if rank else None) + \
        tuple(tables[5:])


def gpu_logits(wl, tables, top_m: int, rank: int, n_eval: int, storage: int = 0, metric: int = 0) -> np.ndarray:
    """Quantise the whole cache with these tables and return the masked logits
    [B, H, n_eval, n_cache] of the first n_eval Queries (scaled by 1/sqrt(d)).
    storage: App. D.1 options (1 = 8-bit group scales, 2 = retention gate);
    metric: 1 ranks the QSAC candidates by the full form (tables[5] is its matrix)."""
    torch, qw = _torch()
    dev = "cuda:0"
    dt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    cfg = qw.make_config(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, rank, top_m, wl.n_cache,
                         wl.dtype, storage, metric)
    mu_k, mu_v, w, u_t, lam = tables[:5]
    T = lambda x, t=dt: torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(dev).to(t)  # noqa: E731
    calib = torch.zeros(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=dev)
    qw.quantwm_calib_pack(cfg, T(mu_k), T(mu_v), T(w, torch.float32), T(u_t) if rank else None,
                          T(lam, torch.float32) if rank else None, calib,
                          m=T(tables[5], torch.float32) if metric else None)
    cache = torch.zeros(qw.quantwm_cache_bytes(cfg), dtype=torch.uint8, device=dev)
    for s0, n in wl.chunks():
        k = T(synth.tensor(wl, "k", n, start=s0))
        v = T(synth.tensor(wl, "v", n, start=s0))
        qw.quantwm_append(cfg, calib, cache, s0, k, v, n)
    q = T(synth.tensor(wl, "q", n_eval))
    lg = torch.empty((wl.batch, wl.heads, n_eval, wl.n_cache), dtype=torch.float32, device=dev)
    qw.quantwm_logits(cfg, calib, cache, wl.n_cache, q, n_eval, wl.q_start, wl.frame_tokens, lg)
    torch.cuda.synchronize()
    return lg.cpu().numpy()


def exact_logits(wl, n_eval: int) -> np.ndarray:
    """fp32 q.k / sqrt(d) of the inputs as the library receives them (rounded to
    the workload's dtype), [B, H, n_eval, n_cache]; masking is left to metrics()."""
    k = synth.round_to(synth.tensor(wl, "k", wl.n_cache), wl.dtype)
    q = synth.round_to(synth.tensor(wl, "q", n_eval), wl.dtype)
    out = np.empty((wl.batch, wl.heads, n_eval, wl.n_cache), np.float32)
    for b in range(wl.batch):
        for h in range(wl.heads):
            out[b, h] = (q[b, :, h, :] @ k[b, :, h, :].T) / np.float32(math.sqrt(wl.head_dim))
    return out


# App. D.1 storage options, applied to the "both" mode
STORAGE = {"i8_scales": 1, "gate": 2, "i8_scales+gate": 3}
# QSAC candidate metric of the "both" mode: Eq. 9 (diagonal) or the full form
METRIC = {"diagonal": 0, "full": 1}


def evaluate(wl, tables, n_eval: int, modes=tuple(MODES), m_sweep=(1, 2, 4, 8), storage=tuple(STORAGE),
             metric=tuple(METRIC)) -> dict:
    exact = exact_logits(wl, n_eval)
    vis = visible_mask(wl, n_eval, wl.n_cache)
    res = {"modes": {}, "m_sweep": {}, "storage": {}, "metric": {}}
    for name in storage:
        (top_m, rank), t = mode_tables(tables, wl, "both")
        res["storage"][name] = metrics(exact, gpu_logits(wl, t, top_m, rank, n_eval, STORAGE[name]), vis)
    for name in metric:
        (top_m, rank), t = mode_tables(tables, wl, "both")
        res["metric"][name] = metrics(exact, gpu_logits(wl, t, top_m, rank, n_eval, metric=METRIC[name]), vis)
    for mode in modes:
        (top_m, rank), t = mode_tables(tables, wl, mode)
        res["modes"][mode] = metrics(exact, gpu_logits(wl, t, top_m, rank, n_eval), vis)
    for m in m_sweep:
        if m > wl.n_centroids:
            continue
        (top_m, rank), t = mode_tables(tables, wl, (m, False, True))
        res["m_sweep"][str(m)] = metrics(exact, gpu_logits(wl, t, top_m, rank, n_eval), vis)
    return res


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--workload", default="mg2-12h", choices=sorted(synth.WORKLOADS))
    ap.add_argument("--n-eval", type=int, default=512, help="Queries of the chunk to evaluate")
    args = ap.parse_args()
    wl = synth.WORKLOADS[args.workload]
    n_eval = min(args.n_eval, wl.n_q)
    res = evaluate(wl, gpu_tables(wl), n_eval)
    res.update({"workload": wl.name, "n_eval": n_eval, "data": "synthetic",
                "modes_def": {k: {"M": v[0] or wl.top_m, "w": "1" if v[1] else "Eq. 8", "r": wl.rank if v[2] else 0}
                              for k, v in MODES.items()}})
    print(json.dumps(res))


if __name__ == "__main__":
    main()
