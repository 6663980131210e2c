"""Calibration epochs (the streaming setting): running Query statistics on the
GPU, recalibration from them, and attention over a cache whose chunks were
appended with different calibration blocks, against the oracle."""
import numpy as np
import pytest
import torch

import harness
import oracle
import synth
from paper_2609_26425_amd import quantwm as qw

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _say(msg):
    print(msg, flush=True)


def _dt(wl):
    return torch.bfloat16 if wl.dtype == "bf16" else torch.float32


def _cfg(wl, metric=0):
    return qw.make_config(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m,
                          wl.n_cache, wl.dtype, wl.storage, metric=metric)


@pytest.mark.parametrize("metric", [0, 1], ids=["diag", "full"])
def test_running_statistics_equal_one_pass(metric):
    # Eq. 6 online: three updates give the fp64 sums of q q^T over all tokens in
    # order (numpy, fp64), and recalibrating from them gives the very block that
    # one-pass calibration over the concatenated history gives (with the full
    # metric, its matrix and the Key search constants derived from it too).
    wl = synth.scaled(synth.WORKLOADS["mg2-12h"], name="stats", heads=3, n_hist=1500)
    cfg = _cfg(wl, metric)
    dt = _dt(wl)
    qh = synth.tensor(wl, "qhist", wl.n_hist)
    qd = torch.from_numpy(qh).to(DEV, dt)
    stats = torch.zeros(qw.quantwm_stats_bytes(cfg), dtype=torch.uint8, device=DEV)
    for s0, s1 in ((0, 700), (700, 701), (701, 1500)):
        qw.quantwm_stats_update(cfg, qd[:, s0:s1].contiguous(), s1 - s0, stats)
    torch.cuda.synchronize()
    count = int(stats[:8].view(torch.int64).item())
    assert count == wl.n_hist
    sums = stats[256:].view(torch.float64).cpu().numpy().reshape(wl.heads, wl.head_dim, wl.head_dim)
    qr = synth.round_to(qh, wl.dtype).astype(np.float64)
    for h in range(wl.heads):
        ref = qr[0, :, h, :].T @ qr[0, :, h, :]
        np.testing.assert_allclose(sums[h], ref, rtol=1e-12, atol=1e-9)
    nc = 880
    k = torch.from_numpy(synth.tensor(wl, "k", nc)).to(DEV, dt)
    v = torch.from_numpy(synth.tensor(wl, "v", nc)).to(DEV, dt)
    ws = torch.empty(qw.quantwm_calibrate_workspace_bytes(cfg, wl.n_hist, nc), dtype=torch.uint8, device=DEV)
    c_epoch = torch.zeros(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=DEV)
    c_once = torch.zeros_like(c_epoch)
    qw.quantwm_calibrate_epoch(cfg, stats, k, v, nc, wl.kmeans_iters, c_epoch, ws)
    qw.quantwm_calibrate(cfg, qd, wl.n_hist, k, v, nc, wl.kmeans_iters, c_once, ws)
    torch.cuda.synchronize()
    assert torch.equal(c_epoch, c_once)
    # a zeroed buffer is the cold start
    cold = torch.zeros_like(stats)
    c_cold = torch.zeros_like(c_epoch)
    qw.quantwm_calibrate_epoch(cfg, cold, k, v, nc, wl.kmeans_iters, c_cold, ws)
    L = qw.quantwm_calib_offsets(cfg)
    w = c_cold.view(wl.heads, L.slab_bytes)[:, L.w:L.w + 4 * wl.head_dim].contiguous().view(torch.float32)
    assert torch.all(w == 1.0)


def _epoch_case(wl, starts, seed_hist):
    """Oracle cache of wl whose chunk e (keys [starts[e], starts[e+1])) is appended
    with tables calibrated on that chunk and on a Query history that grows with e."""
    cfg = oracle.cfg_from_workload(wl)
    k = synth.round_to(synth.tensor(wl, "k", wl.n_cache), wl.dtype)
    v = synth.round_to(synth.tensor(wl, "v", wl.n_cache), wl.dtype)
    qh = synth.round_to(synth.tensor(wl, "qhist", seed_hist * len(starts)), wl.dtype)
    bounds = list(starts) + [wl.n_cache]
    tables, cache = [], oracle.new_cache(cfg)
    for e in range(len(starts)):
        s0, s1 = bounds[e], bounds[e + 1]
        t = oracle.calibrate(cfg, qh[:, : seed_hist * (e + 1)], np.ascontiguousarray(k[:, s0:s1]),
                             np.ascontiguousarray(v[:, s0:s1]), 5)
        oracle.append(cfg, t, cache, s0, np.ascontiguousarray(k[:, s0:s1]), np.ascontiguousarray(v[:, s0:s1]))
        tables.append(t)
    return cfg, k, v, tables, cache


def _run_epochs(wl, starts, n_act, rows, seed_hist=300):
    ocfg, k, v, tables, ocache = _epoch_case(wl, starts, seed_hist)
    cfg = _cfg(wl)
    dt = _dt(wl)
    T = lambda x, t=dt: torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(DEV).to(t)  # noqa: E731
    cb = qw.quantwm_calib_bytes(cfg)
    calibs = torch.zeros(cb * len(starts), dtype=torch.uint8, device=DEV)
    for e, t in enumerate(tables):
        qw.quantwm_calib_pack(cfg, T(t[0]), T(t[1]), T(t[2], torch.float32), T(t[3]) if wl.rank else None,
                              T(t[4], torch.float32) if wl.rank else None, calibs[e * cb:(e + 1) * cb])
    n_pk = wl.n_cache - n_act
    cache = torch.from_numpy(ocache).to(DEV)
    q = synth.round_to(synth.tensor(wl, "q", wl.n_q), wl.dtype)
    qd = T(q)
    ka, va = (T(k[:, n_pk:]), T(v[:, n_pk:])) if n_act else (None, None)
    o_out, o_lse, _ = oracle.attend(ocfg, None, ocache, n_pk, q, wl.q_start, wl.frame_tokens, rows=rows,
                                    k_act=np.ascontiguousarray(k[:, n_pk:]) if n_act else None,
                                    v_act=np.ascontiguousarray(v[:, n_pk:]) if n_act else None,
                                    epochs=list(zip(starts, tables)))
    tol = 2e-2 if wl.dtype == "bf16" else 1e-4
    for mode in ("none", "split", "per-epoch"):
        nb = {"none": 0, "split": qw.quantwm_attend_workspace_bytes(cfg, wl.n_cache, wl.n_q),
              "per-epoch": qw.quantwm_attend_epochs_workspace_bytes(cfg, list(starts), n_pk, n_act, wl.n_q)}[mode]
        if mode != "none" and nb == 0:
            continue
        ws = torch.empty(nb, dtype=torch.uint8, device=DEV) if nb else None
        out = torch.empty_like(qd)
        lse = torch.empty((wl.batch, wl.heads, wl.n_q), dtype=torch.float32, device=DEV)
        _say(f"[gpu] attend_epochs ({mode}) {wl.name}: epochs {list(starts)}, {n_pk} packed + {n_act} exact, "
             f"ws {nb} B")
        qw.quantwm_attend_epochs(cfg, calibs, list(starts), cache, n_pk, ka, va, n_act, qd, wl.n_q, wl.q_start,
                                 wl.frame_tokens, out, lse, ws)
        out2, lse2 = torch.empty_like(out), torch.empty_like(lse)
        qw.quantwm_attend_epochs(cfg, calibs, list(starts), cache, n_pk, ka, va, n_act, qd, wl.n_q, wl.q_start,
                                 wl.frame_tokens, out2, lse2, ws)
        torch.cuda.synchronize()
        assert torch.equal(out, out2) and torch.equal(lse, lse2), f"attend_epochs ({mode}) is not deterministic"
        g = out.float().cpu().numpy()[rows[:, 0], rows[:, 2], rows[:, 1], :]
        gl = lse.cpu().numpy()[rows[:, 0], rows[:, 1], rows[:, 2]]
        err = np.abs(g - o_out)
        assert err.max() <= tol, f"epoch attention max-abs error {err.max():.3g} > {tol}"
        fin = np.isfinite(o_lse)
        assert np.array_equal(np.isfinite(gl), fin)
        assert np.all(np.abs(gl[fin] - o_lse[fin]) <= harness.lse_tol(o_lse[fin]))
        _say(f"[ok] attend_epochs ({mode}) {wl.name}: max-abs {err.max():.3g} "
             f"mean-abs {err.mean():.3g} over {len(rows)} rows")
    # the same cache read as a single epoch is further from the oracle's epochs
    return tables


SMALL_EPOCH = synth.Workload(name="epochs-small", dtype="bf16", batch=1, heads=3, head_dim=128, n_cache=1000,
                             n_q=300, q_start=700, frame_tokens=50, n_centroids=37, group_size=32, rank=12,
                             top_m=3, q_rank=12, n_out=4, out_scale=10.0, n_hist=600, chunk=300, seed=21)
TINY_EPOCH = synth.scaled(synth.WORKLOADS["tiny-f32"], name="epochs-tiny", seed=5)


@pytest.mark.parametrize("wl,starts,n_act", [
    (SMALL_EPOCH, [0, 333, 700], 0),      # boundaries inside tiles (333, 700)
    (SMALL_EPOCH, [0, 333, 640], 150),    # a tile-aligned boundary, then an exact active chunk
    (TINY_EPOCH, [0, 100, 500], 0),       # fp32 path
    (synth.scaled(SMALL_EPOCH, name="epochs-small-i8", storage=1), [0, 333, 700], 0),  # 8-bit group scales
    (synth.scaled(SMALL_EPOCH, name="epochs-small-i8-act", storage=3), [0, 333, 640], 150),  # and an active chunk
    (synth.scaled(TINY_EPOCH, name="epochs-tiny-i8", storage=1), [0, 100, 500], 0),  # fp32 with 8-bit scales
], ids=["bf16-3epochs", "bf16-active", "f32", "bf16-i8", "bf16-i8-gate-active", "f32-i8"])
def test_epoch_attention_small(wl, starts, n_act):
    rows = np.array([(b, h, i) for b in range(wl.batch) for h in range(wl.heads) for i in range(wl.n_q)], np.int32)
    _run_epochs(wl, starts, n_act, rows)


@pytest.mark.timeout(900)
def test_epoch_attention_matrix_game_shape():
    # 5 epochs of one 2,640-token chunk each over the 12-head Matrix-Game shape
    wl = synth.WORKLOADS["mg2-12h"]
    starts = [0, 2640, 5280, 7920, 10560]
    rows = harness.sample_rows(wl, 12, 37)
    _run_epochs(wl, starts, 0, rows, seed_hist=800)


def test_epoch_argument_errors():
    wl = SMALL_EPOCH
    cfg = _cfg(wl)
    buf = torch.zeros(1 << 20, dtype=torch.uint8, device=DEV)
    with pytest.raises(qw.QuantwmError):   # epoch shorter than 64 keys
        qw.quantwm_attend_epochs(cfg, buf, [0, 30], buf, 1000, None, None, 0, buf, 4, 700, 50, buf)
    with pytest.raises(qw.QuantwmError):   # first epoch not at key 0
        qw.quantwm_attend_epochs(cfg, buf, [5, 300], buf, 1000, None, None, 0, buf, 4, 700, 50, buf)
    with pytest.raises(qw.QuantwmError):   # epoch past the packed keys
        qw.quantwm_attend_epochs(cfg, buf, [0, 1000], buf, 1000, None, None, 0, buf, 4, 700, 50, buf)
