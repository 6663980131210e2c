"""Edge and degenerate cases of the method, GPU against the oracle: a single
centroid, zero residuals (scale 0), all-history and all-chunk masks, a
partial single tile, token-causal frames, zero and very large Queries."""
import numpy as np
import pytest

import harness
import synth
import test_parity_gpu as tp

pytestmark = pytest.mark.gpu


def _wl(name, **kw):
    base = dict(name=name, dtype="bf16", batch=1, heads=2, head_dim=128, n_cache=700, n_q=300, q_start=400,
                frame_tokens=50, n_centroids=16, group_size=32, rank=8, top_m=4, q_rank=8, n_out=4, out_scale=10.0,
                n_hist=600, chunk=350, seed=31)
    base.update(kw)
    return synth.Workload(**base)


def _zero_residual(wl):
    # kmeans_iters = 0 keeps the initial centroids, tokens floor(j * nc / Kc) of the
    # calibration chunk; copying them elsewhere gives keys with zero residual
    nc = min(wl.chunk, wl.n_cache)
    seeds = [(j * nc) // wl.n_centroids for j in range(wl.n_centroids)]

    def tf(k, v, q):
        k, v = k.copy(), v.copy()
        for p in range(nc, wl.n_cache, 3):
            j = seeds[p % wl.n_centroids]
            k[:, p], v[:, p] = k[:, j], v[:, j]
        return k, v, q
    return tf


CASES = [
    (_wl("kc1-m4", n_centroids=1, head_dim=64, group_size=16, rank=4, q_rank=4), None),
    (_wl("zero-residual", kmeans_iters=0), "zero_residual"),
    (_wl("history-only", n_cache=500, n_q=64, q_start=500), None),
    (_wl("chunk-only", n_cache=600, n_q=600, q_start=0, frame_tokens=16), None),
    (_wl("one-partial-tile", n_cache=40, n_q=1, q_start=39, frame_tokens=1, chunk=40, n_hist=100), None),
    (_wl("token-causal", frame_tokens=1), None),
    (_wl("zero-query"), "zero_q"),
    (_wl("large-logits", out_scale=10.0), "big_q"),
    # App. D.1 storage options on the degenerate cases: all-zero group steps give
    # sigma = 0 (every step code 0), a single centroid, and a lone partial tile
    (_wl("zero-residual-i8-gate", kmeans_iters=0, storage=3), "zero_residual"),
    (_wl("kc1-i8", n_centroids=1, head_dim=64, group_size=16, rank=4, q_rank=4, storage=1), None),
    (_wl("one-partial-tile-i8-gate", n_cache=40, n_q=1, q_start=39, frame_tokens=1, chunk=40, n_hist=100,
         storage=3), None),
    # the attention producers read binary16 copies of the centroid tables scaled by a
    # power of two: Keys 2^11 times larger put the largest Key centroid components
    # past binary16's range (so the scale is 2^-e with e > 0; the Value tables take
    # e < 0 in every case), and a centroid component
    # of 3e-12 lies below the copy's resolution (it reads as 0 there)
    (_wl("large-keys"), "large_keys"),
    (_wl("tiny-centroid-component"), "tiny_centroid"),
]


def _transform(wl, kind):
    if kind is None:
        return None
    if kind == "zero_residual":
        return _zero_residual(wl)
    if kind == "zero_q":
        return lambda k, v, q: (k, v, np.zeros_like(q))
    if kind == "big_q":
        return lambda k, v, q: (k, v, q * 30.0)
    if kind == "large_keys":
        return lambda k, v, q: (k * 2048.0, v, q)
    if kind == "tiny_centroid":
        return None
    raise ValueError(kind)


def _tables_edit(kind):
    if kind != "tiny_centroid":
        return None

    def edit(tables):
        # one tiny component in centroid 3 of every head's Key and Value tables
        # (a BF16 value, far below 2^-31 of the table's largest magnitude)
        tiny = float(synth.round_to(np.array([3e-12]), "bf16")[0])
        tables[0][..., 3, 5] = tiny
        tables[1][..., 3, 7] = -tiny
    return edit


@pytest.mark.parametrize("wl,kind", CASES, ids=[c[0].name for c in CASES])
def test_edge_case(wl, kind):
    key = (wl.name, 64)
    if key not in tp._cases:
        tp._cases[key] = harness.build_oracle_case(wl, 64, transform=_transform(wl, kind),
                                                   tables_edit=_tables_edit(kind))
    case = tp._cases[key]
    if kind == "large_keys":
        assert np.abs(case.tables[0]).max() > 65504.0, "the Key table should leave binary16's range"
    if kind == "zero_residual":
        import packed
        f = packed.fields(case.cache, case.lay, 0, 0, wl.n_cache)
        assert int((f["k_scale"] == 0).sum()) > 0, "the case should contain zero-scale groups"
        if wl.storage & 1:
            assert int((f["k_sigma"] == 0).sum()) > 0, "the case should contain zero secondary scales"
        if wl.rank:
            assert int((f["k_cscale"] == 0).sum()) > 0, "the case should contain zero coefficient rows"
    tp.run_case(wl, max_sources=64, n_heads_rows=64, row_step=1, logits_rows=wl.n_q)
