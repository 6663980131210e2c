"""The attention entry point that allocates nothing (quantwm_attend_noalloc),
through the C ABI, against quantwm_attend with a caller workspace: two calls in
a row on one static buffer, the second with a smaller input, both with a key
split. Inputs are the oracle's cache and tables (no input comes from the HIP
path); the bar is the bf16 output bar of the parity tests, and bit equality
where both calls split the key range the same way."""
import numpy as np
import pytest
import torch

import harness
import synth

pytestmark = pytest.mark.gpu

from paper_2609_26425_amd import quantwm as qw  # noqa: E402

DEV = "cuda:0"


def _dev(x, dt):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV).to(dt)


def _calib(cfg, tables):
    mu_k, mu_v, w, u_t, lam = tables[:5]
    dt = cfg.torch_dtype
    calib = torch.empty(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=DEV)
    qw.quantwm_calib_pack(cfg, _dev(mu_k, dt), _dev(mu_v, dt), _dev(w, torch.float32), _dev(u_t, dt),
                          _dev(lam, torch.float32), calib)
    return calib


def _run_pair(cfg, calib, cache, q, n_cache, n_q, q_start, F):
    dt = cfg.torch_dtype
    wl_heads, d = cfg.heads, cfg.head_dim
    qd = q[:, :n_q].contiguous()
    out_a = torch.full((cfg.batch, n_q, wl_heads, d), float("nan"), dtype=dt, device=DEV)
    out_b = torch.full_like(out_a, float("nan"))
    lse_a = torch.full((cfg.batch, wl_heads, n_q), float("nan"), dtype=torch.float32, device=DEV)
    lse_b = torch.full_like(lse_a, float("nan"))
    ws_bytes = qw.quantwm_attend_workspace_bytes(cfg, n_cache, n_q)
    assert ws_bytes > 0, "the case must take the key split"
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device=DEV)
    qw.quantwm_attend(cfg, calib, cache, n_cache, qd, n_q, q_start, F, out_a, lse_a, workspace=ws)
    qw.quantwm_attend_noalloc(cfg, calib, cache, n_cache, qd, n_q, q_start, F, out_b, lse_b)
    torch.cuda.synchronize()
    return out_a.float().cpu().numpy(), lse_a.cpu().numpy(), out_b.float().cpu().numpy(), lse_b.cpu().numpy(), ws_bytes


def test_noalloc_matches_attend_with_workspace_on_two_calls():
    wl = synth.scaled(synth.WORKLOADS["mg2-12h"], name="noalloc")
    print(f"noalloc: {wl.name} heads={wl.heads} n_cache={wl.n_cache} n_q={wl.n_q}", flush=True)
    case = harness.build_oracle_case(wl, max_sources=3)
    cfg = qw.make_config(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m,
                         wl.n_cache, wl.dtype)
    calib = _calib(cfg, harness.full_tables(case))
    cache = torch.from_numpy(harness.full_oracle_cache(case)).to(DEV)
    q = _dev(harness.full_inputs(case, "q"), cfg.torch_dtype)
    calls = [(wl.n_cache, wl.n_q, wl.q_start, wl.frame_tokens),   # 13,200 keys, 2,640 Queries
             (6000, 1000, 5000, 500)]                             # then a smaller call on the same buffer
    for n_cache, n_q, q_start, F in calls:
        print(f"noalloc: call n_cache={n_cache} n_q={n_q}", flush=True)
        oa, la, ob, lb, ws_bytes = _run_pair(cfg, calib, cache, q, n_cache, n_q, q_start, F)
        assert np.isfinite(ob).all() and np.isfinite(lb).all()
        assert np.abs(ob - oa).max() <= 2e-2
        assert np.all(np.abs(lb - la) <= 1e-3 * (1 + np.abs(la)))
        if ws_bytes <= qw.ATTEND_NOALLOC_SCRATCH_BYTES:
            # the same split count: the same kernels over the same key ranges
            np.testing.assert_array_equal(ob, oa)
            np.testing.assert_array_equal(lb, la)


def test_noalloc_cuts_a_split_that_exceeds_its_buffer():
    # 40 heads x 1,560 Queries over 60,000 keys: quantwm_attend splits the key
    # range 5 ways (5 partial planes, 162 MB); the static buffer holds 4, so the
    # call takes 4 parts. Inputs: seeded random Keys/Values/Queries calibrated
    # and appended on the GPU (both calls read the same cache).
    H, d, n_cache, n_q = 40, 128, 60000, 1560
    cfg = qw.make_config(1, H, d, 128, 32, 16, 4, n_cache, "bf16")
    g = torch.Generator(device=DEV).manual_seed(7)
    k = torch.randn((1, n_cache, H, d), generator=g, device=DEV).mul_(2.0).to(torch.bfloat16)
    v = torch.randn((1, n_cache, H, d), generator=g, device=DEV).to(torch.bfloat16)
    qh = torch.randn((1, 2048, H, d), generator=g, device=DEV).to(torch.bfloat16)
    q = torch.randn((1, n_q, H, d), generator=g, device=DEV).to(torch.bfloat16)
    calib = torch.empty(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=DEV)
    ws = torch.empty(qw.quantwm_calibrate_workspace_bytes(cfg, 2048, 4680), dtype=torch.uint8, device=DEV)
    qw.quantwm_calibrate(cfg, qh, 2048, k[:, :4680].contiguous(), v[:, :4680].contiguous(), 4680, 3, calib, ws)
    cache = torch.zeros(qw.quantwm_cache_bytes(cfg), dtype=torch.uint8, device=DEV)
    qw.quantwm_append(cfg, calib, cache, 0, k, v, n_cache)
    ws_bytes = qw.quantwm_attend_workspace_bytes(cfg, n_cache, n_q)
    assert ws_bytes > qw.ATTEND_NOALLOC_SCRATCH_BYTES
    print(f"noalloc: cut case, attend workspace {ws_bytes} B", flush=True)
    oa, la, ob, lb, _ = _run_pair(cfg, calib, cache, q, n_cache, n_q, n_cache - n_q, n_q)
    assert np.isfinite(ob).all() and np.isfinite(lb).all()
    assert np.abs(ob - oa).max() <= 2e-2
    assert np.all(np.abs(lb - la) <= 1e-3 * (1 + np.abs(la)))
