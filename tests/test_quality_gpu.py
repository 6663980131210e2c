"""Synthetic quality harness: orderings the method predicts, and its metrics
computed from the library's logits against the same metrics computed from the
oracle's logits (same tables, same inputs)."""
import numpy as np
import pytest

import oracle
import quality
import synth

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)


def _oracle_tables(wl):
    # with the full metric's matrix as a sixth table
    cfg = oracle.cfg_from_workload(wl)
    cfg.metric = oracle.METRIC_FULL
    nc = min(wl.chunk, wl.n_cache)
    k = synth.round_to(synth.tensor(wl, "k", nc), wl.dtype)
    v = synth.round_to(synth.tensor(wl, "v", nc), wl.dtype)
    qh = synth.round_to(synth.tensor(wl, "qhist", wl.n_hist), wl.dtype)
    return oracle.calibrate(cfg, qh, k, v, wl.kmeans_iters)


def _oracle_logits(wl, tables, top_m, rank, n_eval, storage=0, metric=0):
    cfg = oracle.cfg_of(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, rank, top_m, wl.n_cache,
                        wl.dtype == "bf16", storage, metric)
    cache = oracle.new_cache(cfg)
    k = synth.round_to(synth.tensor(wl, "k", wl.n_cache), wl.dtype)
    v = synth.round_to(synth.tensor(wl, "v", wl.n_cache), wl.dtype)
    for s0, n in wl.chunks():
        oracle.append(cfg, tables, cache, s0, np.ascontiguousarray(k[:, s0:s0 + n]),
                      np.ascontiguousarray(v[:, s0:s0 + n]))
    q = synth.round_to(synth.tensor(wl, "q", n_eval), wl.dtype)
    rows = np.array([(b, h, i) for b in range(wl.batch) for h in range(wl.heads) for i in range(n_eval)], np.int32)
    _, _, lg = oracle.attend(cfg, tables, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens, rows=rows,
                             want_logits=True)
    return lg.reshape(wl.batch, wl.heads, n_eval, wl.n_cache)


def test_quality_metrics_match_oracle():
    # f4 parity: every mode's logit MSE and top-1 shift from the library equal
    # those from the oracle on the tiny fp32 workload.
    wl = synth.WORKLOADS["tiny-f32"]
    n_eval = 128
    tables = _oracle_tables(wl)
    exact = quality.exact_logits(wl, n_eval)
    vis = quality.visible_mask(wl, n_eval, wl.n_cache)
    for mode in quality.MODES:
        (top_m, rank), t = quality.mode_tables(tables, wl, mode)
        g = quality.metrics(exact, quality.gpu_logits(wl, t, top_m, rank, n_eval), vis)
        o = quality.metrics(exact, _oracle_logits(wl, t, top_m, rank, n_eval), vis)
        _say(f"[ok] quality {mode}: gpu {g} oracle {o}")
        assert abs(g["logit_mse"] - o["logit_mse"]) <= 1e-3 * o["logit_mse"]
        assert abs(g["top1_shift"] - o["top1_shift"]) <= 2.0 / (wl.batch * wl.heads * n_eval)
    for name, storage in quality.STORAGE.items():
        (top_m, rank), t = quality.mode_tables(tables, wl, "both")
        g = quality.metrics(exact, quality.gpu_logits(wl, t, top_m, rank, n_eval, storage), vis)
        o = quality.metrics(exact, _oracle_logits(wl, t, top_m, rank, n_eval, storage), vis)
        _say(f"[ok] quality both + {name}: gpu {g} oracle {o}")
        assert abs(g["logit_mse"] - o["logit_mse"]) <= 1e-3 * o["logit_mse"]
        assert abs(g["top1_shift"] - o["top1_shift"]) <= 2.0 / (wl.batch * wl.heads * n_eval)
    (top_m, rank), t = quality.mode_tables(tables, wl, "both")
    g = quality.metrics(exact, quality.gpu_logits(wl, t, top_m, rank, n_eval, metric=1), vis)
    o = quality.metrics(exact, _oracle_logits(wl, t, top_m, rank, n_eval, metric=1), vis)
    _say(f"[ok] quality both, full metric: gpu {g} oracle {o}")
    assert abs(g["logit_mse"] - o["logit_mse"]) <= 1e-3 * o["logit_mse"]
    assert abs(g["top1_shift"] - o["top1_shift"]) <= 2.0 / (wl.batch * wl.heads * n_eval)


def test_quality_orderings_on_matrix_game_shape():
    # Sec. 4.2 / Eq. 14-16: PSAC removes the Key error along the dominant Query
    # directions, so it lowers the logit error of Queries from that distribution;
    # with QSAC it is the lowest of the four settings.
    wl = synth.scaled(synth.WORKLOADS["mg2-12h"], name="mg2-4h", heads=4, n_cache=4400, n_q=880, q_start=3520,
                      chunk=880, n_hist=1760)
    res = quality.evaluate(wl, quality.gpu_tables(wl), 256, m_sweep=(1, 4))
    m = res["modes"]
    _say(f"[ok] quality mg2-4h: {m} storage {res['storage']} metric {res['metric']}")
    assert m["psac"]["logit_mse"] < m["qvg"]["logit_mse"]
    assert m["both"]["logit_mse"] < m["qsac"]["logit_mse"]
    assert m["both"]["logit_mse"] < m["qvg"]["logit_mse"]
    assert m["both"]["top1_shift"] <= m["qvg"]["top1_shift"]
    assert res["m_sweep"]["4"]["logit_mse"] == pytest.approx(m["both"]["logit_mse"], rel=1e-12)


def test_qsac_ordering_with_queries_on_the_outlier_channels():
    # Sec. 4.1: QSAC helps where the Queries load the channels whose Key residuals
    # are hard to quantise. Here the dominant Query directions lie on the Key
    # outlier channels (8 of them, x20): QSAC alone lowers the logit MSE below
    # plain nearest-centroid quantisation (QVG), and PSAC, which removes the
    # error along those same directions, lowers it most.
    wl = synth.scaled(synth.WORKLOADS["mg2-12h"], name="mg2-4h-aligned", heads=4, n_cache=2640, n_q=880,
                      q_start=1760, chunk=880, n_hist=1760, q_align=1.0, n_out=8, out_scale=20.0)
    res = quality.evaluate(wl, quality.gpu_tables(wl), 128, m_sweep=(), storage=(), metric=())
    m = res["modes"]
    _say(f"[ok] quality {wl.name}: {m}")
    assert m["qsac"]["logit_mse"] < m["qvg"]["logit_mse"]
    assert m["psac"]["logit_mse"] < m["qsac"]["logit_mse"]
    assert m["both"]["logit_mse"] < m["qsac"]["logit_mse"]
