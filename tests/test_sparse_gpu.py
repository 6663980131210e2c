"""GPU parity of the resident sparse PSAC rows (App. D.1 per-chunk dense or
sparse coefficient layout in the cache that attention reads): the library's
append writes the same row pools, tile directories and overflow counts as the
oracle, and attention over such a cache matches the oracle's, in every form
that reads it. Rows are dropped by planting tokens that equal a centroid of
their head exactly (zero residual, so the PSAC row is zero); the memory the
pools save is reported."""
import numpy as np
import pytest
import torch

import harness
import oracle
import packed
import synth

pytestmark = pytest.mark.gpu

import test_parity_gpu as tp  # noqa: E402
from paper_2609_26425_amd import quantwm as qw  # noqa: E402

DEV = "cuda:0"
_SP, _GATE, _I8 = oracle.STORE_SPARSE, oracle.STORE_GATE, oracle.STORE_SCALE_I8


def _say(msg):
    print(msg, flush=True)


def planted_case(wl, drop_frac, max_sources, seed=5):
    """An OracleCase whose sources drop about drop_frac of their rows (tokens set
    to a centroid after calibration), appended chunk by chunk as on the GPU."""
    sources = harness.sources_for(wl, max_sources)
    S = len(sources)
    stage = wl.coef_stage or wl.chunk
    cfg = oracle.cfg_of(1, S, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m, wl.n_cache,
                        wl.dtype == "bf16", wl.storage, wl.metric, wl.coef_rows, stage)
    k = harness._gen_sources(wl, sources, "k", wl.n_cache)
    v = harness._gen_sources(wl, sources, "v", wl.n_cache)
    q = harness._gen_sources(wl, sources, "q", wl.n_q)
    qh = harness._gen_sources(wl, sources, "qhist", wl.n_hist)
    nc = min(wl.chunk, wl.n_cache)
    tables = oracle.calibrate(cfg, qh, np.ascontiguousarray(k[:, :nc]), np.ascontiguousarray(v[:, :nc]),
                              wl.kmeans_iters)
    r = np.random.default_rng(seed)
    drop = r.random(wl.n_cache) < drop_frac
    for s in range(S):
        for t in np.nonzero(drop)[0]:
            k[0, t, s] = tables[0][0, s, r.integers(wl.n_centroids)]
    cache = oracle.new_cache(cfg)
    coefs, kids, vids, cands = [], [], [], []
    for s0, n in wl.chunks():
        dg = oracle.append(cfg, tables, cache, s0, np.ascontiguousarray(k[:, s0:s0 + n]),
                           np.ascontiguousarray(v[:, s0:s0 + n]), diagnostics=True)
        coefs.append(dg["coef"]); kids.append(dg["k_ids"]); vids.append(dg["v_ids"]); cands.append(dg["cand"])
    diag = {"coef": np.concatenate(coefs, 2), "k_ids": np.concatenate(kids, 2), "v_ids": np.concatenate(vids, 2),
            "cand": np.concatenate(cands, 2)}
    lay = packed.layout(1, S, wl.head_dim, wl.group_size, wl.rank, wl.n_cache, wl.storage, wl.coef_rows, stage)
    bh = wl.batch * wl.heads
    src_of = np.arange(bh) % S
    return harness.OracleCase(wl, sources, src_of, k, v, q, tables, cfg, cache, diag, lay), drop


def gpu_cfg(wl):
    return qw.make_config(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m,
                          wl.n_cache, wl.dtype, wl.storage, wl.metric, wl.coef_rows, wl.coef_stage or wl.chunk)


def run_sparse(wl, drop_frac, max_sources, n_heads_rows, row_step):
    _say(f"[case] {wl.name}: pool {wl.coef_rows or 'one row per slot'}, ~{drop_frac:.0%} rows planted to drop")
    case, drop = planted_case(wl, drop_frac, max_sources)
    cfg = gpu_cfg(wl)
    calib = tp.gpu_calib_from_tables(cfg, harness.full_tables(case))
    g_cache, g_coef = tp.gpu_append_all(wl, cfg, calib, harness.full_inputs(case, "k"), harness.full_inputs(case, "v"))
    st = tp.check_append(case, g_cache, g_coef)
    _say(f"[ok] append {wl.name}: {st}")
    # the directories and overflow counters are exact (a planted token has distance 0
    # to its centroid, so no near-tie decides whether a row is kept)
    lay = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.n_cache, wl.storage,
                        wl.coef_rows, wl.coef_stage or wl.chunk)
    for bh in range(wl.batch * wl.heads):
        s = int(case.src_of[bh])
        gb, gm = packed.directory(g_cache, lay, bh)
        ob, om = packed.directory(case.cache, case.lay, s)
        nt = (wl.n_cache + 63) // 64
        np.testing.assert_array_equal(gb[:nt], ob[:nt])
        np.testing.assert_array_equal(gm[:nt], om[:nt])
        assert packed.overflow(g_cache, lay, bh) == packed.overflow(case.cache, case.lay, s)
    used, dropped = qw.quantwm_coef_pool_usage(cfg, torch.from_numpy(g_cache).to(DEV), wl.n_cache)
    slots = wl.batch * wl.heads * wl.n_cache
    dense_b = qw.quantwm_cache_bytes(tp.gpu_config(synth.scaled(wl, storage=wl.storage & ~_SP)))
    sparse_b = qw.quantwm_cache_bytes(cfg)
    _say(f"[ok] pools {wl.name}: {used} rows for {slots} slots ({1 - used / slots:.1%} fewer), {dropped} without "
         f"room; cache {sparse_b} B against {dense_b} B dense ({1 - sparse_b / dense_b:.1%} smaller)")
    assert used <= slots and (used < 0.8 * slots or drop_frac < 0.2)
    # attention over the oracle's cache, against the oracle, in every form that reads it
    ora_full = harness.full_oracle_cache(case)
    q_full = harness.full_inputs(case, "q")
    rows = harness.sample_rows(wl, n_heads_rows, row_step)
    for split in (False, True):
        nb = qw.quantwm_attend_workspace_bytes(cfg, wl.n_cache, wl.n_q)
        if split and nb == 0:
            continue
        out, lse = tp.gpu_attend(wl, cfg, calib, ora_full, q_full, split)
        out2, lse2 = tp.gpu_attend(wl, cfg, calib, ora_full, q_full, split)
        assert np.array_equal(out, out2) and np.array_equal(lse, lse2), "attend is not deterministic"
        mx, mean = tp.check_attend(case, out, lse, rows)
        _say(f"[ok] attend{' split' if split else ''} {wl.name}: max-abs {mx:.3g} mean-abs {mean:.3g}")
    # and over the library's own cache: the same result (its rows equal the oracle's)
    out_g, _ = tp.gpu_attend(wl, cfg, calib, g_cache, q_full)
    out_o, _ = tp.gpu_attend(wl, cfg, calib, ora_full, q_full)
    assert np.abs(out_g - out_o).max() <= 2e-2
    # the logits hook and the chunk records read slot-addressed rows: refused
    with pytest.raises(qw.QuantwmError):
        qw.quantwm_logits(cfg, calib, torch.from_numpy(g_cache).to(DEV), wl.n_cache,
                          tp.tdev(q_full[:, :4], cfg.torch_dtype), 4, wl.q_start, wl.frame_tokens,
                          torch.empty((wl.batch, wl.heads, 4, wl.n_cache), device=DEV))
    return used, slots


SMALL = synth.Workload(name="sparse-ragged", dtype="bf16", batch=2, heads=3, head_dim=128, n_cache=1000, n_q=300,
                       q_start=700, frame_tokens=50, n_centroids=37, group_size=32, rank=12, top_m=3, q_rank=8,
                       n_out=4, out_scale=10.0, n_hist=500, chunk=300, seed=7, storage=_SP | _GATE)


@pytest.mark.parametrize("wl,frac", [
    (SMALL, 0.35),
    (synth.scaled(SMALL, name="sparse-ragged-i8", storage=_SP | _GATE | _I8), 0.35),
    (synth.scaled(SMALL, name="sparse-nogate", storage=_SP), 0.35),
    (synth.scaled(SMALL, name="sparse-dense-chunks", storage=_SP | _GATE), 0.0),   # every chunk dense
    (synth.scaled(SMALL, name="sparse-pool-overflow", coef_rows=560), 0.35),       # the last chunk spills
    (synth.scaled(synth.WORKLOADS["tiny-f32"], name="sparse-tiny-f32", storage=_SP | _GATE), 0.5),
], ids=["gate", "gate-i8", "no-gate", "dense", "overflow", "f32"])
def test_sparse_rows_small(wl, frac):
    run_sparse(wl, frac, 64, 64, 1)


@pytest.mark.timeout(900)
def test_sparse_rows_lingbot():
    # the 40-head LingBot shape with 35% of the rows dropped, and a pool sized
    # for the rows kept plus one chunk
    base = synth.WORKLOADS["lingbot-40h"]
    wl = synth.scaled(base, name="lingbot-40h-sparse", storage=_SP | _GATE, coef_rows=26000)
    used, slots = run_sparse(wl, 0.35, 3, 6, 37)
    assert used < 0.7 * slots


def test_sparse_active_chunk_and_epochs():
    # the streaming forms read sparse rows too: an exact active chunk after the
    # packed keys, and two calibration epochs (one launch each)
    wl = SMALL
    case, _ = planted_case(wl, 0.35, 64)
    cfg = gpu_cfg(wl)
    calib = tp.gpu_calib_from_tables(cfg, harness.full_tables(case))
    ora_full = torch.from_numpy(harness.full_oracle_cache(case)).to(DEV)
    q_full = harness.full_inputs(case, "q")
    dt = cfg.torch_dtype
    q = tp.tdev(q_full, dt)
    n_act = 200
    n_pk = wl.n_cache - n_act
    k_full, v_full = harness.full_inputs(case, "k"), harness.full_inputs(case, "v")
    ka, va = tp.tdev(np.ascontiguousarray(k_full[:, n_pk:]), dt), tp.tdev(np.ascontiguousarray(v_full[:, n_pk:]), dt)
    rows = harness.sample_rows(wl, 64, 1)
    src_rows = np.array([(0, int(case.src_of[b * wl.heads + h]), i) for b, h, i in rows], np.int32)
    uniq, inv = np.unique(src_rows, axis=0, return_inverse=True)
    o_out, o_lse, _ = oracle.attend(case.cfg, case.tables, case.cache, n_pk, case.q, wl.q_start, wl.frame_tokens,
                                    rows=uniq, k_act=np.ascontiguousarray(case.k[:, n_pk:]),
                                    v_act=np.ascontiguousarray(case.v[:, n_pk:]))
    o_out = o_out[inv.ravel()]
    ws_b = qw.quantwm_attend_active_workspace_bytes(cfg, n_pk, n_act, wl.n_q)
    for ws in (None, torch.empty(max(ws_b, 256), dtype=torch.uint8, device=DEV)):
        out = torch.empty_like(q)
        lse = torch.empty((wl.batch, wl.heads, wl.n_q), dtype=torch.float32, device=DEV)
        qw.quantwm_attend_active(cfg, calib, ora_full, n_pk, ka, va, n_act, q, wl.n_q, wl.q_start, wl.frame_tokens,
                                 out, lse, ws)
        torch.cuda.synchronize()
        g = out.float().cpu().numpy()[rows[:, 0], rows[:, 2], rows[:, 1], :]
        assert np.abs(g - o_out).max() <= 2e-2
    # epochs: the same tables twice (the per-epoch arithmetic is pinned elsewhere);
    # the result equals plain attention over the sparse rows up to the order in
    # which the correction term is summed at the epoch boundary
    cb = qw.quantwm_calib_bytes(cfg)
    calibs = torch.cat([calib, calib])
    out_e = torch.empty_like(q)
    qw.quantwm_attend_epochs(cfg, calibs, [0, 400], ora_full, wl.n_cache, None, None, 0, q, wl.n_q, wl.q_start,
                             wl.frame_tokens, out_e)
    out_p = torch.empty_like(q)
    qw.quantwm_attend(cfg, calib, ora_full, wl.n_cache, q, wl.n_q, wl.q_start, wl.frame_tokens, out_p)
    torch.cuda.synchronize()
    assert cb > 0 and (out_e.float() - out_p.float()).abs().max().item() <= 2e-2
