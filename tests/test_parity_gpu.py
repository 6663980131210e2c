"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bar (ids and codes exact except counted fp32 near-ties; PSAC coefficients
within 1e-4 relative; logits within 1e-3 relative; outputs within 2e-2 max-abs
for bf16). Small cases run the oracle on every head; the benchmark workloads run
the GPU at full size in the benchmark's launch configuration, with every head
replicating one of a few oracle-computed source heads (tests/harness.py).
"""
import math

import numpy as np
import pytest
import torch

import harness
import oracle
import packed
import synth

pytestmark = pytest.mark.gpu

from paper_2609_26425_amd import quantwm as qw  # noqa: E402  (fails loudly if the library is missing)

DEV = "cuda:0"


def _say(msg):
    print(msg, flush=True)


def tdev(x, dtype):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV).to(dtype)


def gpu_config(wl, capacity=None):
    return qw.make_config(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank,
                          wl.top_m, wl.n_cache if capacity is None else capacity, wl.dtype, wl.storage, wl.metric)


def gpu_calib_from_tables(cfg, tables):
    """tables: (mu_k, mu_v, w, u_t, lam[, m]); m is the full metric's matrix."""
    mu_k, mu_v, w, u_t, lam = tables[:5]
    m = tables[5] if len(tables) > 5 else None
    dt = cfg.torch_dtype
    calib = torch.empty(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=DEV)
    qw.quantwm_calib_pack(cfg, tdev(mu_k, dt), tdev(mu_v, dt), tdev(w, torch.float32),
                          tdev(u_t, dt) if cfg.rank > 0 else None, tdev(lam, torch.float32) if cfg.rank > 0 else None,
                          calib, m=tdev(m, torch.float32) if m is not None else None)
    return calib


def gpu_append_all(wl, cfg, calib, k_full, v_full):
    dt = cfg.torch_dtype
    cache = torch.zeros(qw.quantwm_cache_bytes(cfg), dtype=torch.uint8, device=DEV)
    coef = torch.zeros((wl.batch, wl.heads, wl.n_cache, max(wl.rank, 1)), dtype=torch.float32, device=DEV)
    kd, vd = tdev(k_full, dt), tdev(v_full, dt)
    for start, n in wl.chunks():
        kc = kd[:, start:start + n].contiguous()
        vc = vd[:, start:start + n].contiguous()
        co = torch.zeros((wl.batch, wl.heads, n, max(wl.rank, 1)), dtype=torch.float32, device=DEV) \
            if wl.rank > 0 else None
        qw.quantwm_append(cfg, calib, cache, start, kc, vc, n, co)
        if co is not None:
            coef[:, :, start:start + n] = co
    torch.cuda.synchronize()
    return cache.cpu().numpy(), coef[..., :wl.rank].cpu().numpy()


def check_append(case, gpu_cache, gpu_coef):
    wl = case.wl
    lay = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.n_cache, wl.storage,
                         wl.coef_rows, wl.coef_stage or wl.chunk)
    mu_k, mu_v, w = case.tables[0][0], case.tables[1][0], case.tables[2][0]
    lam = case.tables[4][0] if wl.rank > 0 else None
    mfull = case.tables[5][0] if wl.metric == oracle.METRIC_FULL else None
    M = min(wl.top_m, wl.n_centroids)
    stats = {"tokens": 0, "k_ties": 0, "v_ties": 0, "coef_half": 0, "cscale_f16": 0, "gate_ties": 0}
    i8 = bool(wl.storage & oracle.STORE_SCALE_I8)
    gate = bool(wl.storage & oracle.STORE_GATE) and wl.rank > 0
    for bh in range(wl.batch * wl.heads):
        s = int(case.src_of[bh])
        g = packed.fields(gpu_cache, lay, bh, 0, wl.n_cache)
        o = packed.fields(case.cache, case.lay, s, 0, wl.n_cache)
        stats["tokens"] += wl.n_cache
        kmis = np.nonzero(g["k_ids"] != o["k_ids"])[0]
        for t in kmis:
            tie = harness.qsac_near_tie(case.k[0, t, s], mu_k[s], w[s], M) if mfull is None else \
                harness.qsac_near_tie_full(case.k[0, t, s], mu_k[s], mfull[s], M)
            assert tie, f"head {bh} token {t}: K centroid {g['k_ids'][t]} vs oracle {o['k_ids'][t]} is not a near-tie"
        vmis = np.nonzero(g["v_ids"] != o["v_ids"])[0]
        for t in vmis:
            assert harness.nearest_near_tie(case.v[0, t, s], mu_v[s]), \
                f"head {bh} token {t}: V centroid {g['v_ids'][t]} vs oracle {o['v_ids'][t]} is not a near-tie"
        stats["k_ties"] += len(kmis)
        stats["v_ties"] += len(vmis)
        kok = np.ones(wl.n_cache, bool); kok[kmis] = False
        vok = np.ones(wl.n_cache, bool); vok[vmis] = False
        for f in ("k_codes", "k_zp", "k_scale") + (("k_sigma",) if i8 else ()):
            bad = np.nonzero((g[f][kok] != o[f][kok]).reshape(kok.sum(), -1).any(1))[0]
            assert len(bad) == 0, f"head {bh}: {f} differs at tokens {np.nonzero(kok)[0][bad][:8]}"
        for f in ("v_codes", "v_zp", "v_scale") + (("v_sigma",) if i8 else ()):
            bad = np.nonzero((g[f][vok] != o[f][vok]).reshape(vok.sum(), -1).any(1))[0]
            assert len(bad) == 0, f"head {bh}: {f} differs at tokens {np.nonzero(vok)[0][bad][:8]}"
        if wl.rank > 0:
            b, h = divmod(bh, wl.heads)
            Cg = gpu_coef[b, h][kok].astype(np.float64)
            Co = case.diag["coef"][0, s][kok].astype(np.float64)
            tol = 1e-4 * np.abs(Co).max(1) + 1e-7
            err = np.abs(Cg - Co).max(1)
            assert np.all(err <= tol), f"head {bh}: PSAC coefficient error {err.max()} > 1e-4 relative"
            sc_g, sc_o = g["k_cscale"][kok], o["k_cscale"][kok]
            amax = np.abs(Co).max(1).astype(np.float32) / np.float32(127.0)
            if gate:
                # a row kept on one side and zeroed on the other: the keep rule
                # must be at a tie (errors before and after within rounding)
                flip = (sc_g == 0) != (sc_o == 0)
                for t in np.nonzero(flip)[0]:
                    src = g if sc_o[t] == 0 else o
                    sv = float(np.uint16(src["k_cscale"][kok][t]).view(np.float16))
                    e = Co[t] - src["k_coef"][kok][t].astype(np.float64) * sv
                    before = float(np.sum(lam[s].astype(np.float64) * Co[t] ** 2))
                    after = float(np.sum(lam[s].astype(np.float64) * e ** 2))
                    assert abs(after - before) <= 1e-4 * before + 1e-30, f"head {bh}: gate differs off a tie"
                stats["gate_ties"] += int(flip.sum())
                both = ~flip
                Co, sc_g, sc_o, amax = Co[both], sc_g[both], sc_o[both], amax[both]
                kok_rows = np.nonzero(kok)[0][both]
                kok = np.zeros_like(kok)
                kok[kok_rows] = True
                zero = sc_o == 0  # dropped on both sides: all codes 0
                assert not g["k_coef"][kok][zero].any() and not o["k_coef"][kok][zero].any()
            sbad = sc_g != sc_o
            assert np.all(harness.f16_boundary(amax[sbad])), f"head {bh}: coefficient scale differs off a tie"
            stats["cscale_f16"] += int(sbad.sum())
            cg, co_ = g["k_coef"][kok].astype(np.int32), o["k_coef"][kok].astype(np.int32)
            same_scale = ~sbad
            diff = (cg != co_) & same_scale[:, None]
            if diff.any():
                sval = np.array([np.uint16(x).view(np.float16) for x in sc_o], np.float64)
                ratio = Co / np.where(sval > 0, sval, 1.0)[:, None]
                ok = (np.abs(cg - co_) == 1) & harness.near_half(ratio, 1e-3)
                assert np.all(ok[diff]), f"head {bh}: INT8 coefficient codes differ off a .5 tie"
                stats["coef_half"] += int(diff.sum())
    assert stats["k_ties"] + stats["v_ties"] <= max(4, 2e-3 * stats["tokens"]), stats
    return stats


def gpu_attend(wl, cfg, calib, cache_np, q_full, split=False):
    """quantwm_attend without a workspace, or (split=True) with the workspace it
    asks for, which splits the key range when the launch under-fills the GPU."""
    dt = cfg.torch_dtype
    cache = torch.from_numpy(cache_np).to(DEV)
    q = tdev(q_full, dt)
    out = torch.empty_like(q)
    lse = torch.empty((wl.batch, wl.heads, wl.n_q), dtype=torch.float32, device=DEV)
    ws = None
    if split:
        nb = qw.quantwm_attend_workspace_bytes(cfg, wl.n_cache, wl.n_q)
        ws = torch.empty(nb, dtype=torch.uint8, device=DEV)
    qw.quantwm_attend(cfg, calib, cache, wl.n_cache, q, wl.n_q, wl.q_start, wl.frame_tokens, out, lse, ws)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), lse.cpu().numpy()


def check_attend(case, out, lse, rows):
    wl = case.wl
    src_rows = np.array([(0, int(case.src_of[b * wl.heads + h]), i) for b, h, i in rows], np.int32)
    uniq, inv = np.unique(src_rows, axis=0, return_inverse=True)
    o_out, o_lse, _ = oracle.attend(case.cfg, case.tables, case.cache, wl.n_cache, case.q, wl.q_start,
                                    wl.frame_tokens, rows=uniq)
    o_out, o_lse = o_out[inv.ravel()], o_lse[inv.ravel()]
    g_out = out[rows[:, 0], rows[:, 2], rows[:, 1], :]
    g_lse = lse[rows[:, 0], rows[:, 1], rows[:, 2]]
    tol = 2e-2 if wl.dtype == "bf16" else 1e-4
    err = np.abs(g_out - o_out)
    assert err.max() <= tol, f"attention output max-abs error {err.max():.3g} > {tol} (mean {err.mean():.3g})"
    fin = np.isfinite(o_lse)
    assert np.array_equal(np.isfinite(g_lse), fin)
    assert np.all(np.abs(g_lse[fin] - o_lse[fin]) <= harness.lse_tol(o_lse[fin])), \
        f"lse error {np.abs(g_lse[fin] - o_lse[fin]).max():.3g}"
    return float(err.max()), float(err.mean())


def check_logits(case, cfg, calib, cache_np, q_full, n_q_rows, first=0):
    """Logits hook on the n_q_rows Queries from chunk row `first` on, every head
    (full key range)."""
    wl = case.wl
    dt = cfg.torch_dtype
    n_q = min(n_q_rows, wl.n_q - first)
    q = tdev(np.ascontiguousarray(q_full[:, first:first + n_q]), dt)
    cache = torch.from_numpy(cache_np).to(DEV)
    lg = torch.empty((wl.batch, wl.heads, n_q, wl.n_cache), dtype=torch.float32, device=DEV)
    qw.quantwm_logits(cfg, calib, cache, wl.n_cache, q, n_q, wl.q_start, wl.frame_tokens, lg, q_first=first)
    torch.cuda.synchronize()
    lg = lg.cpu().numpy()
    rows = np.array([(0, s, first + i) for s in range(len(case.sources)) for i in range(n_q)], np.int32)
    _, _, o_lg = oracle.attend(case.cfg, case.tables, case.cache, wl.n_cache, case.q, wl.q_start, wl.frame_tokens,
                               rows=rows, want_logits=True)
    worst = 0.0
    for bh in range(wl.batch * wl.heads):
        b, h = divmod(bh, wl.heads)
        s = int(case.src_of[bh])
        for i in range(n_q):
            ref = o_lg[s * n_q + i]
            got = lg[b, h, i]
            vis = np.isfinite(ref)
            assert np.array_equal(vis, np.isfinite(got)), f"mask differs at head {bh} row {first + i}"
            e = np.abs(got[vis] - ref[vis]).max() / max(np.abs(ref[vis]).max(), 1e-30)
            worst = max(worst, e)
            assert e <= 1e-3, f"logits error {e:.3g} at head {bh} row {first + i}"
    return worst


def frame_row_starts(wl, rows):
    """First chunk rows of `rows`-row windows that straddle every frame boundary
    of the Query chunk (and the chunk's first and last rows)."""
    F = wl.frame_tokens
    starts = {0, max(0, wl.n_q - rows)}
    for f in range(1, (wl.n_q + F - 1) // F):
        starts.add(min(max(0, f * F - rows // 2), max(0, wl.n_q - rows)))
    return sorted(starts)


# ------------------------------------------------------------------ cases

RAGGED = synth.Workload(name="ragged", dtype="bf16", batch=2, heads=3, head_dim=128, n_cache=1000, n_q=300,
                        q_start=700, frame_tokens=50, n_centroids=37, group_size=32, rank=12, top_m=3, q_rank=8,
                        n_out=4, out_scale=10.0, n_hist=500, chunk=300, seed=7)
D64 = synth.Workload(name="d64-g16-m8", dtype="bf16", batch=1, heads=2, head_dim=64, n_cache=700, n_q=130,
                     q_start=570, frame_tokens=1, n_centroids=24, group_size=16, rank=20, top_m=8, q_rank=6,
                     n_out=2, out_scale=10.0, n_hist=400, chunk=350, seed=8)
NOPSAC = synth.Workload(name="g64-r0-m1", dtype="bf16", batch=1, heads=2, head_dim=128, n_cache=513, n_q=257,
                        q_start=256, frame_tokens=64, n_centroids=5, group_size=64, rank=0, top_m=1, q_rank=4,
                        n_out=2, out_scale=20.0, n_hist=300, chunk=513, seed=9)

# fp32 at d = 128 (the fp32 matrix-core instances of that width, r = 16), and
# d = 128 with G = 16: eight groups per token, so two zero-point bytes
F32D128 = synth.Workload(name="f32-d128", dtype="f32", batch=1, heads=2, head_dim=128, n_cache=640, n_q=200,
                         q_start=440, frame_tokens=40, n_centroids=16, group_size=32, rank=16, top_m=4, q_rank=8,
                         n_out=4, out_scale=10.0, n_hist=400, chunk=320, seed=12)
D128G16 = synth.Workload(name="d128-g16", dtype="bf16", batch=1, heads=3, head_dim=128, n_cache=650, n_q=190,
                         q_start=460, frame_tokens=38, n_centroids=20, group_size=16, rank=12, top_m=4, q_rank=8,
                         n_out=4, out_scale=10.0, n_hist=400, chunk=325, seed=13)

# BF16 d = 64 with G = 64: the one group spans both lane halves of the BF16
# append kernel (ranges and the 8-bit scales' maximum combined across the pair);
# r = 16 fills the rank padding, so the coefficient rows take the word stores
D64G64 = synth.Workload(name="d64-g64", dtype="bf16", batch=1, heads=2, head_dim=64, n_cache=600, n_q=150,
                        q_start=450, frame_tokens=30, n_centroids=40, group_size=64, rank=16, top_m=4, q_rank=6,
                        n_out=2, out_scale=10.0, n_hist=400, chunk=300, seed=14)

# BF16 appends of 8 tokens (one partial wave per call: most lanes recompute a
# real token and store nothing) and Kc = 16, half of a 32-centroid block
SMALLCHUNK = synth.Workload(name="bf16-chunk8-kc16", dtype="bf16", batch=2, heads=2, head_dim=128, n_cache=200,
                            n_q=40, q_start=160, frame_tokens=8, n_centroids=16, group_size=32, rank=8, top_m=2,
                            q_rank=4, n_out=2, out_scale=10.0, n_hist=200, chunk=8, seed=15)

# BF16 centroid tables too large for LDS (d = 128 with Kc = 256 at r = 32 and
# Kc = 192 at r = 12): the attention instances whose producers read the
# centroid rows from global memory, at small sizes with ragged Query blocks
KC256 = synth.Workload(name="d128-kc256", dtype="bf16", batch=2, heads=2, head_dim=128, n_cache=900, n_q=300,
                       q_start=600, frame_tokens=60, n_centroids=256, group_size=64, rank=32, top_m=4, q_rank=8,
                       n_out=8, out_scale=20.0, n_hist=600, chunk=450, seed=16)
KC192 = synth.Workload(name="d128-kc192", dtype="bf16", batch=1, heads=3, head_dim=128, n_cache=1100, n_q=260,
                       q_start=840, frame_tokens=52, n_centroids=192, group_size=32, rank=12, top_m=4, q_rank=6,
                       n_out=4, out_scale=10.0, n_hist=800, chunk=550, seed=17)

SMALL = [synth.WORKLOADS["tiny-f32"], RAGGED, D64, NOPSAC, F32D128, D128G16, D64G64, SMALLCHUNK, KC256, KC192]

# two workgroups for a key range of 200 or more tiles: the launch splits the
# keys 16 ways (the most the split rule takes), so the combine merges four full
# groups of four partial results per Query (d = 128 and d = 64, BF16 and fp32)
MANYSPLIT = [
    synth.Workload(name="d128-split16", dtype="bf16", batch=1, heads=2, head_dim=128, n_cache=20480,
                   n_q=96, q_start=20384, frame_tokens=32, n_centroids=32, group_size=32, rank=8,
                   top_m=4, q_rank=4, n_out=4, out_scale=10.0, n_hist=1024, chunk=4096, seed=18),
    synth.Workload(name="d64-split16", dtype="bf16", batch=1, heads=2, head_dim=64, n_cache=12800,
                   n_q=40, q_start=12760, frame_tokens=20, n_centroids=24, group_size=16, rank=4,
                   top_m=4, q_rank=4, n_out=2, out_scale=10.0, n_hist=1024, chunk=3200, seed=19),
    synth.Workload(name="f32-d64-split16", dtype="f32", batch=1, heads=2, head_dim=64, n_cache=12800,
                   n_q=40, q_start=12760, frame_tokens=20, n_centroids=24, group_size=32, rank=4,
                   top_m=4, q_rank=4, n_out=2, out_scale=10.0, n_hist=1024, chunk=3200, seed=20),
]
FULL = ["mg2-12h", "lingbot-40h", "batched-4x30h", "rollout-30k", "rollout-60k", "rollout-120k"]

# App. D.1 storage options: 8-bit group scales (I8), the retention gate, both.
# D64 has r = 20 over a 32-rank stride (the unaligned coefficient load), RAGGED
# uneven tiles and batch 2, NOPSAC r = 0 (the gate has nothing to do).
_I8, _GATE = oracle.STORE_SCALE_I8, oracle.STORE_GATE
STORAGE = [synth.scaled(synth.WORKLOADS["tiny-f32"], name="tiny-f32-i8", storage=_I8),
           synth.scaled(RAGGED, name="ragged-i8-gate", storage=_I8 | _GATE),
           synth.scaled(D64, name="d64-i8", storage=_I8),
           synth.scaled(D64, name="d64-gate", storage=_GATE),
           synth.scaled(NOPSAC, name="g64-r0-i8-gate", storage=_I8 | _GATE),
           synth.scaled(D128G16, name="d128-g16-i8-gate", storage=_I8 | _GATE),
           synth.scaled(F32D128, name="f32-d128-i8", storage=_I8),
           synth.scaled(D64G64, name="d64-g64-i8-gate", storage=_I8 | _GATE)]

# The full quadratic QSAC metric (the diagonal-approximation ablation of App. C):
# fp32 d = 64, bf16 with batch 2 and ragged tiles, M = 8 over a small Kc, and
# one LingBot-shaped head pair (Kc = 128, d = 128, G = 32, r = 16) over one frame.
_FULL = oracle.METRIC_FULL
METRIC = [synth.scaled(synth.WORKLOADS["tiny-f32"], name="tiny-f32-fullm", metric=_FULL),
          synth.scaled(RAGGED, name="ragged-fullm", metric=_FULL),
          synth.scaled(D64, name="d64-fullm", metric=_FULL),
          synth.scaled(RAGGED, name="ragged-fullm-i8-gate", metric=_FULL, storage=_I8 | _GATE),
          synth.scaled(synth.WORKLOADS["lingbot-40h"], name="lingbot-2h-fullm", heads=2, n_cache=1560, n_q=520,
                       q_start=1040, frame_tokens=260, chunk=780, n_hist=1560, metric=_FULL)]

_cases = {}


def case_for(wl, max_sources=6):
    key = (wl.name, max_sources)
    if key not in _cases:
        _say(f"[oracle] building case {wl.name} ({max_sources} source heads)")
        _cases[key] = harness.build_oracle_case(wl, max_sources)
    return _cases[key]


def run_case(wl, max_sources, n_heads_rows, row_step, logits_rows):
    _say(f"[case] {wl.name}")
    case = case_for(wl, max_sources)
    cfg = gpu_config(wl)
    tables = harness.full_tables(case)
    calib = gpu_calib_from_tables(cfg, tables)
    _say(f"[gpu] append {wl.name}")
    k_in, v_in = harness.full_inputs(case, "k"), harness.full_inputs(case, "v")
    g_cache, g_coef = gpu_append_all(wl, cfg, calib, k_in, v_in)
    if wl.n_cache * wl.batch * wl.heads <= 1 << 16:
        # append has no order-dependent reduction either: a second pass over the
        # same inputs writes the same bytes
        g2, c2 = gpu_append_all(wl, cfg, calib, k_in, v_in)
        assert np.array_equal(g_cache, g2) and np.array_equal(g_coef, c2), "append is not deterministic"
    st = check_append(case, g_cache, g_coef)
    _say(f"[ok] append {wl.name}: {st}")
    ora_full = harness.full_oracle_cache(case)
    q_full = harness.full_inputs(case, "q")
    rows = harness.sample_rows(wl, n_heads_rows, row_step)
    for split in (False, True):
        nb = qw.quantwm_attend_workspace_bytes(cfg, wl.n_cache, wl.n_q)
        if split and nb == 0:
            continue
        _say(f"[gpu] attend {wl.name} (workspace {nb if split else 0} B)")
        out, lse = gpu_attend(wl, cfg, calib, ora_full, q_full, split)
        # the kernel has no order-dependent reduction: a second call on the same
        # inputs gives the same bits (a read of a matrix-core result before it is
        # written, or a tile-buffer race, shows up here first)
        out2, lse2 = gpu_attend(wl, cfg, calib, ora_full, q_full, split)
        assert np.array_equal(out, out2) and np.array_equal(lse, lse2), "attend is not deterministic"
        mx, mean = check_attend(case, out, lse, rows)
        _say(f"[ok] attend{' split' if split else ''} {wl.name}: max-abs {mx:.3g} mean-abs {mean:.3g} "
             f"over {len(rows)} rows")
    if logits_rows:
        starts = [0] if logits_rows >= wl.n_q else frame_row_starts(wl, logits_rows)
        worst = max(check_logits(case, cfg, calib, ora_full, q_full, logits_rows, first) for first in starts)
        _say(f"[ok] logits {wl.name}: worst relative error {worst:.3g} (rows from {starts})")


@pytest.mark.parametrize("wl", SMALL, ids=[w.name for w in SMALL])
def test_small_parity(wl):
    run_case(wl, max_sources=64, n_heads_rows=64, row_step=1, logits_rows=wl.n_q)


@pytest.mark.parametrize("wl", MANYSPLIT, ids=[w.name for w in MANYSPLIT])
def test_many_key_splits_parity(wl):
    cfg = gpu_config(wl)
    nb = qw.quantwm_attend_workspace_bytes(cfg, wl.n_cache, wl.n_q)
    splits = nb // (wl.batch * wl.heads * wl.n_q * (4 * wl.head_dim + 8))
    _say(f"[case] {wl.name}: workspace {nb} B, {splits} key splits")
    assert splits >= 9, f"expected a split of at least 9 ways, got {splits}"
    run_case(wl, max_sources=64, n_heads_rows=64, row_step=1, logits_rows=32)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", FULL)
def test_full_size_parity(name):
    wl = synth.WORKLOADS[name]
    run_case(wl, max_sources=3, n_heads_rows=6, row_step=37, logits_rows=16)


@pytest.mark.parametrize("wl", STORAGE, ids=[w.name for w in STORAGE])
def test_storage_parity(wl):
    run_case(wl, max_sources=64, n_heads_rows=64, row_step=1, logits_rows=wl.n_q)


@pytest.mark.parametrize("wl", METRIC, ids=[w.name for w in METRIC])
def test_full_metric_parity(wl):
    run_case(wl, max_sources=64, n_heads_rows=64, row_step=3, logits_rows=64)


@pytest.mark.timeout(900)
def test_storage_full_size_parity():
    wl = synth.scaled(synth.WORKLOADS["mg2-12h"], name="mg2-12h-i8-gate", storage=_I8 | _GATE)
    run_case(wl, max_sources=3, n_heads_rows=6, row_step=37, logits_rows=16)



# ------------------------------------------------------------ calibration

def _gpu_calibrate(case):
    wl = case.wl
    cfg = gpu_config(wl)
    dt = cfg.torch_dtype
    nc = min(wl.chunk, wl.n_cache)
    qh = harness._gen_sources(wl, case.sources, "qhist", wl.n_hist)
    src = {"q": qh, "k": np.ascontiguousarray(case.k[:, :nc]), "v": np.ascontiguousarray(case.v[:, :nc])}
    full = {}
    for key, arr in src.items():
        o = np.empty((wl.batch, arr.shape[1], wl.heads, wl.head_dim), np.float32)
        for bh in range(wl.batch * wl.heads):
            b, h = divmod(bh, wl.heads)
            o[b, :, h, :] = arr[0, :, case.src_of[bh], :]
        full[key] = tdev(o, dt)
    calib = torch.zeros(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=DEV)
    ws = torch.empty(qw.quantwm_calibrate_workspace_bytes(cfg, wl.n_hist, nc), dtype=torch.uint8, device=DEV)
    qw.quantwm_calibrate(cfg, full["q"], wl.n_hist, full["k"], full["v"], nc, wl.kmeans_iters, calib, ws)
    torch.cuda.synchronize()
    return cfg, calib.cpu().numpy()


def _slab_field(cfg, buf, bh, name, count, dtype):
    L = qw.quantwm_calib_offsets(cfg)
    off = bh * L.slab_bytes + getattr(L, name)
    nbytes = count * np.dtype(dtype).itemsize
    return np.frombuffer(buf[off:off + nbytes].tobytes(), dtype=dtype)


def _check_search_planes(cfg, buf, bh, K, d):
    """The BF16 planes of the Key search constants: the first two truncate, the
    third is the remainder, and their sum is a_k exactly."""
    a = _slab_field(cfg, buf, bh, "a_k", K * d, np.float32)
    pl = _slab_field(cfg, buf, bh, "a_k3", 3 * K * d, np.uint16).reshape(3, K * d)
    p = (pl.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    np.testing.assert_array_equal(p[0] + p[1] + p[2], a.astype(np.float64), err_msg=f"a_k planes head {bh}")
    np.testing.assert_array_equal(pl[0], a.view(np.uint32) >> 16, err_msg=f"first plane head {bh}")
    r1 = a - p[0].astype(np.float32)
    np.testing.assert_array_equal(pl[1], r1.view(np.uint32) >> 16, err_msg=f"second plane head {bh}")


@pytest.mark.parametrize("name", ["tiny-f32", "ragged", "mg2-12h"])
def test_calibrate_parity(name):
    wl = {"ragged": RAGGED}.get(name) or synth.WORKLOADS[name]
    case = case_for(wl, 64 if name != "mg2-12h" else 3)
    cfg, buf = _gpu_calibrate(case)
    d, K, r = wl.head_dim, wl.n_centroids, wl.rank
    bf = wl.dtype == "bf16"
    for bh in range(wl.batch * wl.heads):
        s = int(case.src_of[bh])
        if bf:
            mk = _slab_field(cfg, buf, bh, "mu_k", K * d, np.uint16).astype(np.uint32) << 16
            mv = _slab_field(cfg, buf, bh, "mu_v", K * d, np.uint16).astype(np.uint32) << 16
            mk, mv = mk.view(np.float32), mv.view(np.float32)
        else:
            mk = _slab_field(cfg, buf, bh, "mu_k", K * d, np.float32)
            mv = _slab_field(cfg, buf, bh, "mu_v", K * d, np.float32)
        np.testing.assert_array_equal(mk.reshape(K, d), case.tables[0][0, s], err_msg=f"mu_k head {bh}")
        np.testing.assert_array_equal(mv.reshape(K, d), case.tables[1][0, s], err_msg=f"mu_v head {bh}")
        w = _slab_field(cfg, buf, bh, "w", d, np.float32)
        np.testing.assert_array_equal(w, case.tables[2][0, s], err_msg=f"w head {bh}")
        if bf:
            _check_search_planes(cfg, buf, bh, K, d)
        if r > 0:
            lam = _slab_field(cfg, buf, bh, "lam", r, np.float32)
            np.testing.assert_allclose(lam, case.tables[4][0, s], rtol=1e-6)
            if bf:
                u = (_slab_field(cfg, buf, bh, "u_t", r * d, np.uint16).astype(np.uint32) << 16).view(np.float32)
            else:
                u = _slab_field(cfg, buf, bh, "u_t", r * d, np.float32)
            u = u.reshape(r, d).astype(np.float64)
            uo = case.tables[3][0, s].astype(np.float64)
            tol = 2.0 ** -8 if bf else 1e-5
            assert np.all(np.abs(u - uo) <= tol * np.abs(uo) + 1e-6), f"U_r head {bh}"
    _say(f"[ok] calibrate {name}")


def test_calibrate_full_metric_parity():
    # the block carries the oracle's Mn exactly (same fp64 sums and division),
    # and the identity at cold start
    wl = METRIC[1]
    case = case_for(wl, 64)
    cfg, buf = _gpu_calibrate(case)
    d = wl.head_dim
    for bh in range(wl.batch * wl.heads):
        s = int(case.src_of[bh])
        m = _slab_field(cfg, buf, bh, "m", d * d, np.float32).reshape(d, d)
        np.testing.assert_array_equal(m, case.tables[5][0, s], err_msg=f"m head {bh}")
        np.testing.assert_array_equal(np.diag(m), _slab_field(cfg, buf, bh, "w", d, np.float32))
        if wl.dtype == "bf16":
            _check_search_planes(cfg, buf, bh, wl.n_centroids, d)  # a_k = -2 Mn mu here
    k = tdev(synth.tensor(wl, "k", 64), cfg.torch_dtype)
    calib = torch.zeros(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=DEV)
    ws = torch.empty(qw.quantwm_calibrate_workspace_bytes(cfg, 0, 64), dtype=torch.uint8, device=DEV)
    qw.quantwm_calibrate(cfg, None, 0, k, k, 64, 2, calib, ws)
    torch.cuda.synchronize()
    cold = calib.cpu().numpy()
    for bh in range(wl.batch * wl.heads):
        assert np.array_equal(_slab_field(cfg, cold, bh, "m", d * d, np.float32).reshape(d, d),
                              np.eye(d, dtype=np.float32))
    _say("[ok] calibrate full metric")


def test_calibrate_cold_start():
    wl = synth.WORKLOADS["tiny-f32"]
    cfg = gpu_config(wl)
    k = tdev(synth.tensor(wl, "k", 64), torch.float32)
    calib = torch.zeros(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=DEV)
    ws = torch.empty(qw.quantwm_calibrate_workspace_bytes(cfg, 0, 64), dtype=torch.uint8, device=DEV)
    qw.quantwm_calibrate(cfg, None, 0, k, k, 64, 3, calib, ws)
    torch.cuda.synchronize()
    buf = calib.cpu().numpy()
    for bh in range(wl.heads):
        assert np.all(_slab_field(cfg, buf, bh, "w", wl.head_dim, np.float32) == 1.0)
        assert not _slab_field(cfg, buf, bh, "u_t", wl.rank * wl.head_dim, np.float32).any()


# ------------------------------------------------------------ edge cases

def test_empty_calls_are_noops():
    wl = RAGGED
    case = case_for(wl, 64)
    cfg = gpu_config(wl)
    calib = gpu_calib_from_tables(cfg, harness.full_tables(case))
    cache = torch.zeros(qw.quantwm_cache_bytes(cfg), dtype=torch.uint8, device=DEV)
    k = torch.zeros((wl.batch, 1, wl.heads, wl.head_dim), dtype=torch.bfloat16, device=DEV)
    qw.quantwm_append(cfg, calib, cache, 0, k, k, 0)
    out = torch.zeros_like(k)
    qw.quantwm_attend(cfg, calib, cache, 0, k, 0, 0, 1, out)
    torch.cuda.synchronize()
    assert not cache.any()


def test_attend_empty_cache_gives_zero_and_neg_inf_lse():
    wl = RAGGED
    case = case_for(wl, 64)
    cfg = gpu_config(wl)
    calib = gpu_calib_from_tables(cfg, harness.full_tables(case))
    cache = torch.zeros(qw.quantwm_cache_bytes(cfg), dtype=torch.uint8, device=DEV)
    q = tdev(harness.full_inputs(case, "q")[:, :40], torch.bfloat16)
    out = torch.ones_like(q)
    lse = torch.zeros((wl.batch, wl.heads, 40), dtype=torch.float32, device=DEV)
    qw.quantwm_attend(cfg, calib, cache, 0, q, 40, 0, 1, out, lse)
    torch.cuda.synchronize()
    assert not out.float().any() and torch.isneginf(lse).all()


def test_capacity_and_argument_errors():
    wl = RAGGED
    cfg = gpu_config(wl)
    calib = torch.zeros(qw.quantwm_calib_bytes(cfg), dtype=torch.uint8, device=DEV)
    cache = torch.zeros(qw.quantwm_cache_bytes(cfg), dtype=torch.uint8, device=DEV)
    k = torch.zeros((wl.batch, 10, wl.heads, wl.head_dim), dtype=torch.bfloat16, device=DEV)
    with pytest.raises(qw.QuantwmError) as e:
        qw.quantwm_append(cfg, calib, cache, wl.n_cache - 5, k, k, 10)
    assert e.value.status == qw.ERR_CAPACITY
    with pytest.raises(qw.QuantwmError) as e:
        qw.quantwm_attend(cfg, calib, cache, 10, k, 10, 11, 1, k)
    assert e.value.status == qw.ERR_INVALID_ARG


# ----------------------------------------- BF16 active chunk (packed history + exact chunk)

def _active_case(wl, max_sources, n_heads_rows, row_step):
    """Packed history = the first n_cache - n_act tokens; the last n_act tokens
    (the chunk being generated) enter exactly. Runs with no workspace (one
    launch), with a split workspace, and with the two-part workspace (packed
    whole tiles through the plain kernel, the rest through the general one,
    merged by log-sum-exp); each against the oracle."""
    case = case_for(wl, max_sources)
    cfg = gpu_config(wl)
    calib = gpu_calib_from_tables(cfg, harness.full_tables(case))
    n_act = min(wl.chunk, wl.n_cache // 3)
    n_pk = wl.n_cache - n_act
    dt = cfg.torch_dtype
    cache = torch.from_numpy(harness.full_oracle_cache(case)).to(DEV)
    k_full, v_full = harness.full_inputs(case, "k"), harness.full_inputs(case, "v")
    k_act = tdev(np.ascontiguousarray(k_full[:, n_pk:]), dt)
    v_act = tdev(np.ascontiguousarray(v_full[:, n_pk:]), dt)
    q = tdev(harness.full_inputs(case, "q"), dt)
    rows = harness.sample_rows(wl, n_heads_rows, row_step)
    src_rows = np.array([(0, int(case.src_of[b * wl.heads + h]), i) for b, h, i in rows], np.int32)
    uniq, inv = np.unique(src_rows, axis=0, return_inverse=True)
    o_out, o_lse, _ = oracle.attend(case.cfg, case.tables, case.cache, n_pk, case.q, wl.q_start, wl.frame_tokens,
                                    rows=uniq, k_act=np.ascontiguousarray(case.k[:, n_pk:]),
                                    v_act=np.ascontiguousarray(case.v[:, n_pk:]))
    o_out, o_lse = o_out[inv.ravel()], o_lse[inv.ravel()]
    tol = 2e-2 if wl.dtype == "bf16" else 1e-4
    for mode in ("none", "split", "two-part"):
        nb = {"none": 0, "split": qw.quantwm_attend_workspace_bytes(cfg, wl.n_cache, wl.n_q),
              "two-part": qw.quantwm_attend_active_workspace_bytes(cfg, n_pk, n_act, wl.n_q)}[mode]
        if mode != "none" and nb == 0:
            continue
        split = mode != "none"
        ws = torch.empty(nb, dtype=torch.uint8, device=DEV) if nb else None
        out = torch.empty_like(q)
        lse = torch.empty((wl.batch, wl.heads, wl.n_q), dtype=torch.float32, device=DEV)
        _say(f"[gpu] attend_active {wl.name}: {n_pk} packed + {n_act} exact keys, workspace {nb} B")
        qw.quantwm_attend_active(cfg, calib, cache, n_pk, k_act, v_act, n_act, q, wl.n_q, wl.q_start,
                                 wl.frame_tokens, out, lse, ws)
        out2, lse2 = torch.empty_like(out), torch.empty_like(lse)
        qw.quantwm_attend_active(cfg, calib, cache, n_pk, k_act, v_act, n_act, q, wl.n_q, wl.q_start,
                                 wl.frame_tokens, out2, lse2, ws)
        torch.cuda.synchronize()
        assert torch.equal(out, out2) and torch.equal(lse, lse2), f"attend_active ({mode}) is not deterministic"
        g = out.float().cpu().numpy()[rows[:, 0], rows[:, 2], rows[:, 1], :]
        gl = lse.cpu().numpy()[rows[:, 0], rows[:, 1], rows[:, 2]]
        err = np.abs(g - o_out)
        assert err.max() <= tol, f"active-chunk attention max-abs error {err.max():.3g} > {tol}"
        fin = np.isfinite(o_lse)
        assert np.array_equal(np.isfinite(gl), fin)
        assert np.all(np.abs(gl[fin] - o_lse[fin]) <= harness.lse_tol(o_lse[fin]))
        _say(f"[ok] attend_active ({mode}) {wl.name}: max-abs {err.max():.3g} "
             f"mean-abs {err.mean():.3g} over {len(rows)} rows")


@pytest.mark.parametrize("wl", SMALL, ids=[w.name for w in SMALL])
def test_active_chunk_small(wl):
    _active_case(wl, 64, 64, 1)


@pytest.mark.parametrize("wl", STORAGE, ids=[w.name for w in STORAGE])
def test_active_chunk_storage(wl):
    # App. D.1 storage options (8-bit group scales with their FP16 secondary
    # scale, the retention gate) beside a BF16 active chunk, in every form
    _active_case(wl, 64, 64, 1)


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["lingbot-40h", "rollout-30k", "lingbot-40h-i8"])
def test_active_chunk_full(name):
    wl = synth.scaled(synth.WORKLOADS["lingbot-40h"], name=name, storage=_I8) if name.endswith("-i8") \
        else synth.WORKLOADS[name]
    _active_case(wl, 3, 6, 37)
