"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test names the passage it follows. The pins are library routines (numpy,
torch, scipy, scikit-learn), closed forms, hand-computed values and brute force
on tiny inputs. A plausible mistake anywhere in the oracle should fail one of
them.
"""
import math

import numpy as np
import pytest
import torch

import oracle
import synth


def rng(seed=0):
    return np.random.default_rng(seed)


# ----------------------------------------------------------------- formats

def test_round_bf16_matches_torch():
    # BF16 storage of centroids and U_r (App. D.1): RNE, checked against torch's cast.
    r = rng(1)
    x = np.concatenate([r.standard_normal(4000) * 10.0 ** r.integers(-6, 6, 4000),
                        np.array([1.0 + 2 ** -8, 1.0 + 3 * 2 ** -8, -(1.0 + 2 ** -8), 0.0, 3e-39, -1e-40])])
    x = x.astype(np.float32)
    want = torch.from_numpy(x).to(torch.bfloat16).to(torch.float64).numpy()
    got = np.array([oracle.round_bf16(float(v)) for v in x])
    np.testing.assert_array_equal(got, want)


def test_round_f16_matches_numpy():
    # FP16 group and row scales (App. D.1), including subnormals and ties.
    r = rng(2)
    x = np.concatenate([r.standard_normal(4000) * 10.0 ** r.integers(-9, 5, 4000),
                        np.array([1.0 + 2 ** -11, 1.0 + 3 * 2 ** -11, 2 ** -25, 3 * 2 ** -25, 65504.0, 6e-8])])
    x = x.astype(np.float32)
    want = x.astype(np.float16)
    got = np.array([oracle.round_f16(float(v)) for v in x])
    np.testing.assert_array_equal(got, want.astype(np.float64))
    bits = np.array([oracle.f16_bits(float(v)) for v in want.astype(np.float64)], np.uint16)
    np.testing.assert_array_equal(bits, want.view(np.uint16))
    back = np.array([oracle.f16_value(int(b)) for b in bits])
    np.testing.assert_array_equal(back, want.astype(np.float64))


# --------------------------------------------------- INT2 residual (Eq. 1-4)

def test_int2_zero_residual_reconstructs_centroid():
    # Eq. 4 with r = 0: khat = mu exactly, all codes and the zero-point 0.
    mu = synth.round_to(rng(3).standard_normal(32) * 3, "bf16")
    codes, zp, sc, xhat = oracle.int2_group(mu, mu)
    assert not codes.any() and zp == 0 and sc == 0
    np.testing.assert_array_equal(xhat, mu)


def test_int2_hand_example_ties_to_even():
    # Range [-1, 2] gives s = 1 and z = 1 (Eq. 2); 0.5 rounds to 0 (ties to even).
    mu = np.zeros(4, np.float32)
    x = np.array([-1.0, 0.5, 2.0, 0.0], np.float32)
    codes, zp, sc, xhat = oracle.int2_group(x, mu)
    assert list(codes) == [0, 1, 3, 1] and zp == 1
    assert sc == np.float16(1.0).view(np.uint16)
    np.testing.assert_array_equal(xhat, [-1.0, 0.0, 2.0, 0.0])


def test_int2_range_contains_zero():
    # All-positive residuals: the 0-extended range keeps z = 0 and q = round(r / s).
    mu = np.zeros(4, np.float32)
    x = np.array([0.2, 0.9, 0.6, 0.3], np.float32)
    codes, zp, sc, _ = oracle.int2_group(x, mu)
    s = np.float32(np.float32(0.9) / np.float32(3.0)).astype(np.float16).astype(np.float32)
    assert zp == 0 and sc == np.float16(s).view(np.uint16)
    assert list(codes) == [int(np.clip(np.rint(v / s), 0, 3)) for v in x]


@pytest.mark.parametrize("seed", range(6))
def test_int2_grid_round_trip(seed):
    # Values already on an INT2 grid (power-of-two scale, both end levels present)
    # come back bit-exactly with the same codes, zero-point and scale.
    r = rng(100 + seed)
    G = 32
    s = 2.0 ** int(r.integers(-4, 3))
    z = int(r.integers(0, 4))
    q = r.integers(0, 4, G)
    q[0], q[1] = 0, 3
    mu = (r.integers(-64, 64, G) / 16.0).astype(np.float32)
    x = (mu.astype(np.float64) + s * (q - z)).astype(np.float32)
    assert np.array_equal(x.astype(np.float64), mu.astype(np.float64) + s * (q - z))
    codes, zp, sc, xhat = oracle.int2_group(x, mu)
    assert zp == z and list(codes) == list(q)
    assert sc == np.float16(s).view(np.uint16)
    np.testing.assert_array_equal(xhat, x)


def _levels_check(x, mu, codes, zp, sc, xhat):
    s16 = np.uint16(sc).view(np.float16).astype(np.float64)
    r = x.astype(np.float64) - mu.astype(np.float64)
    lo, hi = min(0.0, r.min()), max(0.0, r.max())
    s = (hi - lo) / 3.0
    if s16 == 0:
        return
    levels = s16 * (np.arange(4) - zp)
    dist = np.abs(r[:, None] - levels[None, :])
    best = dist.min(axis=1)
    chosen = dist[np.arange(len(r)), codes]
    # the chosen level is the nearest one, up to fp32 rounding of r / s
    assert np.all(chosen <= best + 1e-5 * s16 + 1e-30)
    # error bound: half a step plus the FP16 rounding slack of the scale
    err = np.abs(xhat.astype(np.float64) - x.astype(np.float64))
    ulp = np.spacing(np.abs(xhat).astype(np.float32)).astype(np.float64)
    assert np.all(err <= s16 / 2 + 3 * abs(s - s16) + ulp + 1e-12)


def test_int2_nearest_level_brute_force():
    r = rng(5)
    for _ in range(300):
        n = int(r.choice([4, 16, 32, 64]))
        mu = synth.round_to(r.standard_normal(n), "bf16")
        x = synth.round_to(mu + r.standard_normal(n) * 10.0 ** r.uniform(-3, 1), "bf16")
        _levels_check(x, mu, *oracle.int2_group(x, mu))


def test_int2_widrow_noise_model():
    # Eq. 11: for residuals spread evenly inside each step, E[e^2] ~ step^2 / 12.
    # The group's own min and max sit at a fixed offset from the grid (they set
    # the range), so the statistic is over the other values of each group.
    r = rng(6)
    num = den = 0.0
    for _ in range(4000):
        x = r.uniform(-1.0, 1.0, 32).astype(np.float32)
        mu = np.zeros(32, np.float32)
        codes, zp, sc, xhat = oracle.int2_group(x, mu)
        s16 = float(np.uint16(sc).view(np.float16))
        e = xhat.astype(np.float64) - x
        keep = np.ones(32, bool)
        keep[[np.argmin(x), np.argmax(x)]] = False
        num += float(np.sum(e[keep] ** 2))
        den += keep.sum() * s16 * s16 / 12.0
    assert abs(num / den - 1.0) < 0.03


# ------------------------------------------------------------ QSAC (Eq. 9-12)

W_HAND = np.array([1.0, 2.0, 0.5, 1.0], np.float32)
K_HAND = np.array([1.0, 0.0, 0.0, 0.0], np.float32)
MU_HAND = np.array([[3.0, 2.0, 0.0, 0.0],     # d_Q 12,     S 0
                    [1.0, 0.5, 0.0, 0.0],     # d_Q 0.5,    S 0.75
                    [1.0, 0.0, 0.5, 0.5],     # d_Q 0.375,  S 0
                    [1.0, 0.25, 0.5, -0.25]],  # d_Q 0.3125, S 1.03125
                   np.float32)


@pytest.mark.parametrize("m,z_want,cand_want", [(1, 3, [3]), (2, 2, [3, 2]), (3, 2, [3, 2, 1]),
                                                (4, 0, [3, 2, 1, 0])])
def test_qsac_hand_example(m, z_want, cand_want):
    # Hand-computed Eq. 9 distances and Eq. 12 scores with G = 2 (W = [3, 1.5]):
    # the nearest centroid is not the best-scoring one, and the S tie between
    # ids 0 and 2 goes to the lower id.
    z, cand = oracle.qsac_assign(K_HAND, MU_HAND, W_HAND, 2, m)
    assert z == z_want and list(cand) == cand_want


def test_qsac_m1_is_weighted_nearest_scipy():
    # M = 1: QSAC reduces to the nearest centroid under the Eq. 9 distance,
    # checked against scipy's weighted squared Euclidean distance.
    from scipy.spatial.distance import cdist
    r = rng(7)
    d, kc = 64, 16
    mu = synth.round_to(r.standard_normal((kc, d)) * 2, "bf16")
    w = (r.uniform(0.1, 3.0, d)).astype(np.float32)
    agree = 0
    for _ in range(200):
        k = synth.round_to(mu[r.integers(kc)] + r.standard_normal(d), "bf16")
        dist = cdist(k[None].astype(np.float64), mu.astype(np.float64), "sqeuclidean",
                     w=w.astype(np.float64))[0]
        z, _ = oracle.qsac_assign(k, mu, w, 32, 1)
        srt = np.sort(dist)
        if srt[1] - srt[0] > 1e-4 * srt[0]:
            assert z == int(np.argmin(dist))
            agree += 1
    assert agree > 190


def test_qsac_m1_unit_weights_is_kmeans_assignment():
    # M = 1 and w = 1 is the plain K-means assignment of QVG (Eq. 3).
    from scipy.cluster.vq import vq
    r = rng(8)
    d, kc = 32, 8
    mu = synth.round_to(r.standard_normal((kc, d)) * 3, "bf16")
    x = synth.round_to(mu[r.integers(kc, size=300)] + r.standard_normal((300, d)), "bf16")
    codes, _ = vq(x.astype(np.float64), mu.astype(np.float64))
    got = [oracle.qsac_assign(v, mu, np.ones(d, np.float32), 32, 1)[0] for v in x]
    got_n = [oracle.nearest(v, mu) for v in x]
    assert np.array_equal(got, codes) and np.array_equal(got_n, codes)


def test_qsac_candidates_are_top_m_and_exhaustive_limit():
    # The candidate set is the M smallest Eq. 9 distances; with M = Kc the
    # choice equals the exhaustive argmin of Eq. 12 (fp64 brute force).
    from scipy.spatial.distance import cdist
    r = rng(9)
    d, kc, G = 64, 16, 16
    mu = synth.round_to(r.standard_normal((kc, d)), "bf16")
    w = r.uniform(0.2, 2.0, d).astype(np.float32)
    Wg = w.astype(np.float64).reshape(-1, G).sum(1)
    for _ in range(100):
        k = synth.round_to(mu[r.integers(kc)] + 0.7 * r.standard_normal(d), "bf16")
        dist = cdist(k[None].astype(np.float64), mu.astype(np.float64), "sqeuclidean", w=w.astype(np.float64))[0]
        z4, cand = oracle.qsac_assign(k, mu, w, G, 4)
        srt = np.sort(dist)
        if srt[4] - srt[3] > 1e-4 * srt[3]:
            assert set(cand) == set(np.argsort(dist)[:4])
        res = k[None].astype(np.float64) - mu.astype(np.float64)
        rg = res.reshape(kc, -1, G)
        S = ((rg.max(-1) - rg.min(-1)) ** 2 * Wg[None]).sum(-1)
        zall, _ = oracle.qsac_assign(k, mu, w, G, kc)
        s2 = np.sort(S)
        if s2[1] - s2[0] > 1e-4 * max(s2[0], 1e-30):
            assert zall == int(np.argmin(S))
        assert S[z4] == S[list(cand)].min() or abs(S[z4] - S[list(cand)].min()) <= 1e-5 * S[z4]


def _spd(r, d, cond=20.0):
    """A random symmetric positive-definite matrix with mean diagonal 1 (fp32)."""
    q, _ = np.linalg.qr(r.standard_normal((d, d)))
    ev = np.exp(np.linspace(0.0, math.log(cond), d))
    m = (q * ev[None, :]) @ q.T
    return (m / np.trace(m) * d).astype(np.float32)


def _clear_gap(dist, m, rel=1e-4):
    srt = np.sort(dist)
    return m >= len(dist) or srt[m] - srt[m - 1] > rel * abs(srt[m - 1]) + 1e-12


def test_full_metric_candidates_are_mahalanobis_top_m():
    # App. C ablation: the full quadratic form (k - mu)^T M (k - mu) is the squared
    # Mahalanobis distance with inverse covariance M (scipy's cdist).
    from scipy.spatial.distance import cdist
    r = rng(21)
    d, kc, G = 64, 16, 16
    m = _spd(r, d)
    w = np.diag(m).astype(np.float32)
    mu = synth.round_to(r.standard_normal((kc, d)), "bf16")
    checked = 0
    for _ in range(100):
        k = synth.round_to(mu[r.integers(kc)] + 0.7 * r.standard_normal(d), "bf16")
        dist = cdist(k[None].astype(np.float64), mu.astype(np.float64), "mahalanobis",
                     VI=m.astype(np.float64))[0] ** 2
        _, cand = oracle.qsac_assign_full(k, mu, m, w, G, 4)
        if _clear_gap(dist, 4):
            assert set(cand) == set(np.argsort(dist)[:4])
            checked += 1
    assert checked > 90


def test_full_metric_with_a_diagonal_matrix_is_eq9():
    # With M diagonal the full form is the Eq. 9 distance with w = diag(M): the
    # candidate lists and the choice equal those of plain QSAC.
    r = rng(22)
    d, kc, G = 64, 32, 32
    w = r.uniform(0.1, 3.0, d).astype(np.float32)
    m = np.diag(w).astype(np.float32)
    mu = synth.round_to(r.standard_normal((kc, d)) * 2, "bf16")
    for _ in range(100):
        k = synth.round_to(mu[r.integers(kc)] + r.standard_normal(d), "bf16")
        dist = ((k.astype(np.float64) - mu) ** 2 * w).sum(1)
        zf, cf = oracle.qsac_assign_full(k, mu, m, w, G, 4)
        zd, cd = oracle.qsac_assign(k, mu, w, G, 4)
        if _clear_gap(dist, 4) and all(_clear_gap(np.sort(dist)[:4], i) for i in range(1, 4)):
            assert list(cf) == list(cd) and zf == zd


def test_full_metric_rank_one_is_nearest_along_the_direction():
    # M = u u^T gives (u.(k - mu))^2: the candidates are the centroids whose
    # projections on u are nearest to k's (a one-dimensional nearest neighbour).
    r = rng(23)
    d, kc, G = 32, 16, 16
    u = r.standard_normal(d)
    u /= np.linalg.norm(u)
    m = np.outer(u, u).astype(np.float32)
    w = np.diag(m).astype(np.float32)
    mu = synth.round_to(r.standard_normal((kc, d)), "bf16")
    checked = 0
    for _ in range(100):
        k = synth.round_to(r.standard_normal(d), "bf16")
        gap = np.abs(mu.astype(np.float64) @ u - k.astype(np.float64) @ u)
        _, cand = oracle.qsac_assign_full(k, mu, m, w, G, 3)
        if _clear_gap(gap ** 2, 3, 1e-3):
            assert set(cand) == set(np.argsort(gap)[:3])
            checked += 1
    assert checked > 80


def test_full_metric_is_rotation_invariant():
    # Rotating Keys, centroids and the metric together (k -> Qk, mu -> Q mu,
    # M -> Q M Q^T) keeps every full-form distance, so the candidate list is the
    # same; the diagonal form has no such invariance.
    r = rng(24)
    d, kc, G = 32, 16, 16
    m = _spd(r, d, cond=50.0)
    q, _ = np.linalg.qr(r.standard_normal((d, d)))
    mu = r.standard_normal((kc, d)).astype(np.float32)
    mu_r = (mu.astype(np.float64) @ q.T).astype(np.float32)
    m_r = (q @ m.astype(np.float64) @ q.T).astype(np.float32)
    w, w_r = np.diag(m).copy(), np.diag(m_r).copy()
    same = differ_diag = 0
    for _ in range(100):
        k = (mu[r.integers(kc)] + 0.8 * r.standard_normal(d)).astype(np.float32)
        k_r = (k.astype(np.float64) @ q.T).astype(np.float32)
        e = k.astype(np.float64) - mu
        dist = np.einsum("jc,cd,jd->j", e, m.astype(np.float64), e)
        if not all(_clear_gap(np.sort(dist)[:5], i, 1e-3) for i in range(1, 5)):
            continue
        _, c0 = oracle.qsac_assign_full(k, mu, m, w, G, 4)
        _, c1 = oracle.qsac_assign_full(k_r, mu_r, m_r, w_r, G, 4)
        assert list(c0) == list(c1)
        same += 1
        _, d0 = oracle.qsac_assign(k, mu, w, G, 4)
        _, d1 = oracle.qsac_assign(k_r, mu_r, w_r, G, 4)
        differ_diag += list(d0) != list(d1)
    assert same > 50 and differ_diag > 0


# ------------------------------------------------------------- calibration

def _small_workload(**kw):
    base = dict(name="t", dtype="f32", batch=1, heads=2, head_dim=32, n_cache=256, n_q=64,
                q_start=192, frame_tokens=16, n_centroids=8, group_size=16, rank=4, top_m=4,
                q_rank=4, n_out=2, out_scale=10.0, n_hist=2000, chunk=64, seed=11)
    base.update(kw)
    return synth.Workload(**base)


def test_eigh_matches_numpy():
    # Eq. 15 eigenpairs against LAPACK via numpy.linalg.eigh.
    r = rng(10)
    for n in (4, 17, 64):
        a = r.standard_normal((n, n))
        a = a @ a.T / n
        lam, vt = oracle.eigh(a)
        ref = np.linalg.eigh(a)[0][::-1]
        np.testing.assert_allclose(lam, ref, rtol=1e-11, atol=1e-12)
        np.testing.assert_allclose(vt @ vt.T, np.eye(n), atol=1e-12)
        np.testing.assert_allclose(a @ vt.T, vt.T * lam[None, :], atol=1e-10)
        for i in range(n):  # sign rule: largest-magnitude entry positive
            assert vt[i, np.argmax(np.abs(vt[i]))] > 0


def test_calibrate_sensitivity_and_basis():
    # Eq. 6 and Eq. 8: w has mean 1 and follows diag(M); Eq. 15: U_r spans the
    # top-r eigenvectors of M (numpy eigh), the eigenvalues match.
    wl = _small_workload()
    cfg = oracle.cfg_from_workload(wl)
    qh = synth.tensor(wl, "qhist", wl.n_hist)
    k = synth.tensor(wl, "k", 256)
    v = synth.tensor(wl, "v", 256)
    mu_k, mu_v, w, u_t, lam = oracle.calibrate(cfg, qh, k, v, 5)
    for h in range(wl.heads):
        q = qh[0, :, h, :].astype(np.float64)
        M = q.T @ q / q.shape[0]
        np.testing.assert_allclose(w[0, h].sum(), wl.head_dim, rtol=1e-5)
        np.testing.assert_allclose(w[0, h], np.diag(M) / np.trace(M) * wl.head_dim, rtol=1e-6)
        ev, vec = np.linalg.eigh(M)
        np.testing.assert_allclose(lam[0, h], ev[::-1][: wl.rank], rtol=1e-6)
        U = u_t[0, h].astype(np.float64).T
        P_ref = vec[:, ::-1][:, : wl.rank] @ vec[:, ::-1][:, : wl.rank].T
        np.testing.assert_allclose(U @ U.T, P_ref, atol=1e-6)


def test_calibrate_synthetic_closed_form():
    # Queries N(0, I) + 5 A u with A orthonormal of rank rq: E[M] = I + 25 A A^T,
    # so rq eigenvalues near 26, the rest near 1, and top-r energy 26r/(25r+d)
    # (the "top directions hold most Query energy" observation of Sec. 4.2).
    wl = _small_workload(head_dim=64, rank=4, q_rank=4, n_hist=20000, heads=1)
    cfg = oracle.cfg_from_workload(wl)
    qh = synth.tensor(wl, "qhist", wl.n_hist)
    k = synth.tensor(wl, "k", 64)
    _, _, w, u_t, lam = oracle.calibrate(cfg, qh, k, k, 0)
    assert np.all(np.abs(lam[0, 0] - 26.0) < 2.0)
    q = qh[0, :, 0, :].astype(np.float64)
    energy = lam[0, 0].sum() / np.trace(q.T @ q / q.shape[0])
    assert abs(energy - 26 * 4 / (25 * 4 + 64)) < 0.02
    _, _, a = synth._head_params(wl, 0, 0)
    s = np.linalg.svd(a.T @ u_t[0, 0].astype(np.float64).T, compute_uv=False)
    assert s.min() > 0.99  # principal angles between span(U_r) and span(A) near 0


def test_calibrate_cold_start():
    # Initialisation of historical statistics: no history -> w = 1 and PSAC off.
    wl = _small_workload()
    cfg = oracle.cfg_from_workload(wl)
    k = synth.tensor(wl, "k", 64)
    _, _, w, u_t, lam = oracle.calibrate(cfg, None, k, k, 2)
    assert np.all(w == 1.0) and not u_t.any() and not lam.any()


def test_calibrate_full_metric_matrix():
    # The full metric's matrix is Eq. 6's M over the mean of its diagonal: its
    # diagonal is exactly w (Eq. 8), it is symmetric, it matches numpy's M up to
    # that scale, and at cold start it is the identity.
    wl = _small_workload()
    cfg = oracle.cfg_from_workload(wl)
    cfg.metric = oracle.METRIC_FULL
    qh = synth.tensor(wl, "qhist", wl.n_hist)
    k = synth.tensor(wl, "k", 256)
    mu_k, _, w, _, _, m = oracle.calibrate(cfg, qh, k, k, 2)
    for h in range(wl.heads):
        assert np.array_equal(np.diag(m[0, h]), w[0, h])
        assert np.array_equal(m[0, h], m[0, h].T)
        q = qh[0, :, h, :].astype(np.float64)
        M = q.T @ q / q.shape[0]
        np.testing.assert_allclose(m[0, h], M / np.trace(M) * wl.head_dim, rtol=1e-5, atol=1e-6)
    *_, m0 = oracle.calibrate(cfg, None, k, k, 2)
    assert np.array_equal(m0[0, 0], np.eye(wl.head_dim, dtype=np.float32))


def test_append_full_metric_uses_each_heads_matrix():
    # The append path ranks each head's Keys with that head's matrix: its ids and
    # candidates equal QSAC with the full form per token, and the candidate
    # lists differ from the Eq. 9 ones.
    wl = _small_workload(heads=2, n_centroids=16)
    cfg = oracle.cfg_from_workload(wl, capacity=128)
    cfg.metric = oracle.METRIC_FULL
    r = rng(25)
    tables = list(oracle.calibrate(cfg, synth.tensor(wl, "qhist", 500), synth.tensor(wl, "k", 128),
                                   synth.tensor(wl, "v", 128), 3))
    tables[5] = np.stack([np.stack([_spd(r, wl.head_dim, 200.0) for _ in range(2)])])
    tables[2] = np.ascontiguousarray(np.diagonal(tables[5], axis1=2, axis2=3))
    k = synth.tensor(wl, "k", 128)
    v = synth.tensor(wl, "v", 128)
    cache = oracle.new_cache(cfg)
    got = oracle.append(cfg, tables, cache, 0, k, v, diagnostics=True)
    diff = 0
    for h in range(2):
        for t in range(128):
            z, cand = oracle.qsac_assign_full(k[0, t, h], tables[0][0, h], tables[5][0, h], tables[2][0, h],
                                              wl.group_size, wl.top_m)
            assert got["k_ids"][0, h, t] == z and list(got["cand"][0, h, t]) == list(cand)
            _, cd = oracle.qsac_assign(k[0, t, h], tables[0][0, h], tables[2][0, h], wl.group_size, wl.top_m)
            diff += list(cd) != list(cand)
    assert diff > 0
    with pytest.raises(RuntimeError):
        oracle.append(cfg, tables[:5], oracle.new_cache(cfg), 0, k, v)


def test_kmeans_matches_sklearn_lloyd():
    # Eq. 3 centroids: Lloyd iterations from the same initial tokens agree with
    # scikit-learn's Lloyd K-means on well-separated fp32 data.
    from sklearn.cluster import KMeans
    r = rng(12)
    d, kc, n = 16, 4, 400
    centers = r.standard_normal((kc, d)) * 20
    x = (centers[r.integers(kc, size=n)] + r.standard_normal((n, d))).astype(np.float32)
    wl = _small_workload(head_dim=d, n_centroids=kc, group_size=16, rank=0, heads=1)
    cfg = oracle.cfg_from_workload(wl)
    xt = x[None, :, None, :]
    mu_k, _, _, _, _ = oracle.calibrate(cfg, None, xt, xt, 8)
    init = x[[(j * n) // kc for j in range(kc)]].astype(np.float64)
    km = KMeans(n_clusters=kc, init=init, n_init=1, max_iter=8, tol=0.0, algorithm="lloyd").fit(x.astype(np.float64))
    np.testing.assert_allclose(mu_k[0, 0], km.cluster_centers_, rtol=1e-5, atol=1e-5)


# -------------------------------------------------------- PSAC and attention

def _encoded(wl, with_hist=True, n_new=None):
    cfg = oracle.cfg_from_workload(wl)
    qh = synth.tensor(wl, "qhist", wl.n_hist) if with_hist else None
    k = synth.tensor(wl, "k", wl.n_cache)
    v = synth.tensor(wl, "v", wl.n_cache)
    tables = oracle.calibrate(cfg, qh, k[:, : wl.chunk], v[:, : wl.chunk], 5)
    cache = oracle.new_cache(cfg)
    diag = oracle.append(cfg, tables, cache, 0, k, v, diagnostics=True)
    q = synth.tensor(wl, "q", wl.n_q)
    return cfg, tables, cache, k, v, q, diag


def _sdpa(q, K, V, mask):
    qt = torch.from_numpy(q)[None]
    return torch.nn.functional.scaled_dot_product_attention(
        qt, torch.from_numpy(K)[None], torch.from_numpy(V)[None],
        attn_mask=torch.from_numpy(mask)[None])[0].numpy()


def _mask(wl, n_cache):
    i = np.arange(wl.n_q)[:, None]
    j = np.arange(n_cache)[None, :]
    return (j < wl.q_start) | ((j - wl.q_start) // wl.frame_tokens <= i // wl.frame_tokens)


def test_psac_rank0_is_plain_dequantised_attention():
    # r = 0: attention over the dequantised cache only (Eq. 4 + Eq. 5), against
    # torch's SDPA in fp64 on the decoded Keys and Values.
    wl = _small_workload(rank=0)
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    out, lse, _ = oracle.attend(cfg, tables, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    for h in range(wl.heads):
        k0, _, vh = oracle.decode(cfg, tables, cache, 0, h, wl.n_cache)
        k0 = k0.astype(np.float32).astype(np.float64)
        ref = _sdpa(q[0, :, h, :].astype(np.float64), k0, vh, _mask(wl, wl.n_cache))
        np.testing.assert_allclose(out[h * wl.n_q:(h + 1) * wl.n_q], ref, atol=1e-10)


def test_psac_full_rank_recovers_exact_logits():
    # r = d with the unquantised coefficients C = E U (Eq. 16) and an fp32
    # orthonormal U: Eq. 17 restores the fp32 logits q.k.
    wl = _small_workload(rank=32, head_dim=32, group_size=16)
    cfg, tables, cache, k, v, q, diag = _encoded(wl)
    rows = np.array([(0, h, i) for h in range(wl.heads) for i in range(0, wl.n_q, 7)], np.int32)
    _, _, logits = oracle.attend(cfg, tables, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens,
                                 rows=rows, coef_override=diag["coef"], want_logits=True)
    for n, (b, h, i) in enumerate(rows):
        exact = (k[b, :, h, :].astype(np.float64) @ q[b, i, h, :].astype(np.float64)) / math.sqrt(wl.head_dim)
        vis = np.isfinite(logits[n])
        assert vis.sum() > 0
        scale = np.abs(exact[vis]).max()
        assert np.abs(logits[n][vis] - exact[vis]).max() <= 1e-5 * scale


def test_psac_projection_identity_and_distortion_drop():
    # Eq. 14-16: with C = E U_r, U_r^T (E - C U_r^T)^T = 0, and the expected
    # distortion drops by exactly sum_k lambda_k |E u_k|^2.
    wl = _small_workload(rank=8, head_dim=32, group_size=16)
    cfg, tables, cache, k, v, q, diag = _encoded(wl)
    qh = synth.tensor(wl, "qhist", wl.n_hist)
    for h in range(wl.heads):
        k0, _, _ = oracle.decode(cfg, tables, cache, 0, h, wl.n_cache)
        E = k[0, :, h, :].astype(np.float64) - k0
        U = tables[3][0, h].astype(np.float64).T
        C = diag["coef"][0, h].astype(np.float64)
        np.testing.assert_allclose(C, E @ U, rtol=1e-6, atol=1e-6 * np.abs(E @ U).max())
        qq = qh[0, :, h, :].astype(np.float64)
        M = qq.T @ qq / qq.shape[0]
        D = lambda X: np.trace(X @ M @ X.T)  # noqa: E731
        Er = E - (E @ U) @ U.T
        assert np.abs(Er @ U).max() < 1e-6 * np.abs(E).max()  # U is fp32-rounded
        lam, vec = np.linalg.eigh(M)
        top = vec[:, ::-1][:, : wl.rank]
        drop_closed = sum(lam[::-1][j] * np.sum((E @ top[:, j]) ** 2) for j in range(wl.rank))
        # U is the oracle's fp32 copy of the same eigenvectors: tight but not exact
        assert abs((D(E) - D(Er)) - drop_closed) <= 1e-4 * drop_closed


def test_logit_error_identity_monte_carlo():
    # Eq. 7: E_q[(q^T e)^2] = e^T M e, with M the historical second moment.
    wl = _small_workload(head_dim=32, n_hist=20000)
    qh = synth.tensor(wl, "qhist", wl.n_hist)[0, :, 0, :].astype(np.float64)
    e = rng(13).standard_normal(32)
    M = qh.T @ qh / qh.shape[0]
    assert abs(np.mean((qh @ e) ** 2) / (e @ M @ e) - 1.0) < 1e-12


def test_attend_explicit_reconstruction_fp32():
    # Eq. 17 both ways: the factored (q U) c correction equals attention over the
    # explicitly reconstructed Khat = Khat_0 + C U_r^T (torch SDPA, fp64).
    wl = _small_workload(rank=4)
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    out, lse, _ = oracle.attend(cfg, tables, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    for h in range(wl.heads):
        k0, ch, vh = oracle.decode(cfg, tables, cache, 0, h, wl.n_cache)
        U = tables[3][0, h].astype(np.float64)
        qh = q[0, :, h, :].astype(np.float64)
        # the oracle rounds q U_r to the table type (fp32 here): ~1e-7 relative
        Khat = k0 + ch @ U
        ref = _sdpa(qh, Khat, vh, _mask(wl, wl.n_cache))
        got = out[h * wl.n_q:(h + 1) * wl.n_q]
        assert np.abs(got - ref).max() < 1e-5


def test_attend_uniform_logits_give_mean_value():
    # q = 0: every visible logit is 0, so O is the mean of the visible Values and
    # lse = ln(#visible) (closed form).
    wl = _small_workload(rank=4)
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    qz = np.zeros_like(q)
    out, lse, _ = oracle.attend(cfg, tables, cache, wl.n_cache, qz, wl.q_start, wl.frame_tokens)
    mask = _mask(wl, wl.n_cache)
    for h in range(wl.heads):
        _, _, vh = oracle.decode(cfg, tables, cache, 0, h, wl.n_cache)
        for i in range(0, wl.n_q, 5):
            vis = mask[i]
            np.testing.assert_allclose(out[h * wl.n_q + i], vh[vis].mean(0), atol=1e-12)
            np.testing.assert_allclose(lse[h * wl.n_q + i], math.log(vis.sum()), atol=1e-12)


def test_attend_masked_keys_do_not_contribute():
    # Block-causal visibility: editing Keys/Values that a row cannot see leaves it unchanged.
    wl = _small_workload(rank=4)
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    rows = np.array([(0, 1, 3)], np.int32)
    out1, lse1, _ = oracle.attend(cfg, tables, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens, rows=rows)
    k2, v2 = k.copy(), v.copy()
    first_hidden = wl.q_start + wl.frame_tokens  # row 3 sees only frame 0 of the chunk
    k2[:, first_hidden:] *= -3.0
    v2[:, first_hidden:] += 5.0
    cache2 = oracle.new_cache(cfg)
    oracle.append(cfg, tables, cache2, 0, k2, v2)
    out2, lse2, _ = oracle.attend(cfg, tables, cache2, wl.n_cache, q, wl.q_start, wl.frame_tokens, rows=rows)
    np.testing.assert_array_equal(out1, out2)
    np.testing.assert_array_equal(lse1, lse2)


# ---------------------------------------------------------------- storage

def test_token_bytes_and_paper_compression():
    # App. D.1 storage: 4 codes per byte, uint8 ids, INT2 zero-points, FP16 group
    # scales (the library's default), INT8 PSAC rows with an FP16 scale. At the paper's setting
    # (d = 128, G = 64, r = 8) K+V take 86 B per token-head against 512 B in BF16:
    # 5.95x, close to the reported best case of 6.20x (Sec. 5.5).
    cfg = oracle.cfg_of(1, 1, 128, 256, 64, 8, 4, 64, True)
    kb, vb = oracle.token_bytes(cfg)
    assert (kb, vb) == (32 + 1 + 1 + 4 + 10, 32 + 1 + 1 + 4)
    ratio = 512 / (kb + vb)
    assert abs(ratio - 5.95) < 0.01 and abs(ratio / 6.20 - 1) < 0.05
    for d, G, r, want in [(128, 32, 8, (52, 42)), (128, 32, 16, (60, 42)), (128, 64, 32, (72, 38)),
                          (64, 32, 4, (28, 22))]:
        assert oracle.token_bytes(oracle.cfg_of(1, 1, d, 16, G, r, 4, 64, True)) == want


def test_psac_rank_bits_match_the_rank_sweep():
    # T9 context: dense INT8 rows cost 8 bits per rank per Key token-head, so
    # going from r = 8 to r = 16 adds 64 bits over the 2d = 256 K and V elements:
    # 0.25 bits per element, within 3% of the 0.2569 reported on Causal-Forcing.
    kb8, vb8 = oracle.token_bytes(oracle.cfg_of(1, 1, 128, 128, 32, 8, 4, 64, True))
    kb16, vb16 = oracle.token_bytes(oracle.cfg_of(1, 1, 128, 128, 32, 16, 4, 64, True))
    dbits = 8 * ((kb16 + vb16) - (kb8 + vb8)) / 256
    assert dbits == 0.25 and abs(dbits / 0.2569 - 1) < 0.03


def test_token_bytes_with_8bit_group_scales():
    # App. D.1: group scales as 8-bit codes plus one FP16 secondary scale per
    # token-head, so ng group scales take ng + 2 bytes instead of 2 ng.
    for d, G, r in [(128, 32, 16), (128, 64, 8), (128, 16, 0), (64, 32, 4)]:
        ng = d // G
        cfg = oracle.cfg_of(1, 1, d, 16, G, r, 4, 64, True, oracle.STORE_SCALE_I8)
        v = d // 4 + 1 + (ng + 3) // 4 + ng + 2
        assert oracle.token_bytes(cfg) == (v + (r + 2 if r else 0), v)


# ------------------------------------- App. D.1 storage refinements (NEXT f3)

def test_scales_i8_hand_example():
    # t = (0.3, 0.15, 0, 1.2): sigma = FP16(1.2 / 255) = FP16(0.0047059) =
    # 1234 * 2^-18 (binary16 0x1CD2; 1233.6 units of 2^-18 round up), and
    # c = RN(t / sigma) = RN(63.73, 31.87, 0, 254.92) = (64, 32, 0, 255).
    t = np.array([0.3, 0.15, 0.0, 1.2], np.float32)
    sig, codes, steps = oracle.scales_i8(t)
    assert sig == 0x1CD2
    assert list(codes) == [64, 32, 0, 255]
    sigma = 1234.0 * 2.0 ** -18
    np.testing.assert_array_equal(steps.astype(np.float64), sigma * np.array([64, 32, 0, 255]))


def test_scales_i8_invariants():
    # For any steps: the largest gets code 255 (sigma is max / 255 within FP16
    # rounding), every decoded step lies within sigma / 2 of its step, zero steps
    # get code 0, and scaling all steps by 2^k scales sigma by 2^k and leaves the
    # codes unchanged (binary rounding commutes with powers of two while sigma
    # stays a normal binary16 number, as it does for these ranges).
    r = rng(21)
    for _ in range(500):
        ng = int(r.choice([1, 2, 4, 8]))
        t = (10.0 ** r.uniform(-1, 1.5, ng)).astype(np.float32)
        t[r.random(ng) < 0.2] = 0.0
        sig, codes, steps = oracle.scales_i8(t)
        if not t.any():
            assert sig == 0 and not codes.any()
            continue
        sigma = float(np.uint16(sig).view(np.float16))
        assert codes[np.argmax(t)] == 255
        assert np.all(np.abs(steps.astype(np.float64) - t) <= sigma / 2 * (1 + 1e-6))
        assert np.all(codes[t == 0] == 0)
        k = int(r.integers(-2, 4))
        sig2, codes2, _ = oracle.scales_i8((t * np.float32(2.0 ** k)).astype(np.float32))
        assert float(np.uint16(sig2).view(np.float16)) == sigma * 2.0 ** k
        np.testing.assert_array_equal(codes2, codes)
    sig, codes, steps = oracle.scales_i8(np.zeros(4, np.float32))
    assert sig == 0 and not codes.any() and not steps.any()


def test_int2_quantise_with_the_fp16_step_is_the_group_quantiser():
    # Eq. 1-2 with the stored step: given the FP16 step, the quantiser with a
    # given step reproduces the pinned FP16 group quantiser bit for bit.
    r = rng(22)
    for _ in range(200):
        n = int(r.choice([16, 32, 64]))
        mu = synth.round_to(r.standard_normal(n), "bf16")
        x = synth.round_to(mu + r.standard_normal(n) * 10.0 ** r.uniform(-3, 1), "bf16")
        codes, zp, sc, xhat = oracle.int2_group(x, mu)
        step = float(np.uint16(sc).view(np.float16))
        c2, z2, x2 = oracle.int2_quantise(x, mu, step)
        assert z2 == zp
        np.testing.assert_array_equal(c2, codes)
        np.testing.assert_array_equal(x2, xhat)


def test_keep_row_cases():
    # App. D.1 retention: keep a row only when sum lam (C - chat)^2 < sum lam C^2.
    lam = np.array([2.0, 1.0], np.float32)
    # exact codes: no error left
    assert oracle.keep_row(np.array([1.0, -0.5], np.float32), np.array([2, -1]), 0.5, lam)
    # hand example: codes (1, -1) at scale 1 leave 1 * (0.5)^2 = 0.25 < 2 + 0.25
    assert oracle.keep_row(np.array([1.0, -0.5], np.float32), np.array([1, -1]), 1.0, lam)
    # a zero row, or zero eigenvalues, never lowers the error
    assert not oracle.keep_row(np.zeros(2, np.float32), np.zeros(2), 1.0, lam)
    assert not oracle.keep_row(np.array([1.0, -0.5], np.float32), np.array([2, -1]), 0.5, np.zeros(2, np.float32))
    # the wrong sign doubles the error: 2 * (1 + 1)^2 + (0.5 + 0.5)^2 > 2.25
    assert not oracle.keep_row(np.array([1.0, -0.5], np.float32), np.array([-1, 1]), 1.0, lam)
    # the eigenvalues weight the ranks: moving error from a heavy rank to a light
    # one helps (10 -> 1), the other way round it hurts (1 -> 10)
    C = np.array([1.0, 0.0], np.float32)
    assert oracle.keep_row(C, np.array([1, 1]), 1.0, np.array([10.0, 1.0], np.float32))
    assert not oracle.keep_row(C, np.array([1, 1]), 1.0, np.array([1.0, 10.0], np.float32))


def test_append_8bit_scales_decode_within_half_a_step():
    # Eq. 1-4 with the App. D.1 8-bit scales: the packed fields decode to steps
    # sigma * c_g, every code picks the nearest level of its group's grid, and the
    # decoded Key is within half a step of the input (plus fp32 rounding).
    import packed
    wl = _small_workload(rank=4, storage=oracle.STORE_SCALE_I8)
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    lay = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity, wl.storage)
    assert lay["total"] == oracle.cache_bytes(cfg)
    G, ng = wl.group_size, wl.head_dim // wl.group_size
    for h in range(wl.heads):
        f = packed.fields(cache, lay, h, 0, wl.n_cache)
        k0, _, vh = oracle.decode(cfg, tables, cache, 0, h, wl.n_cache)
        for name, x, xhat, mu_t in (("k", k[0, :, h], k0, tables[0][0, h]), ("v", v[0, :, h], vh, tables[1][0, h])):
            sigma = f[f"{name}_sigma"].view(np.float16).astype(np.float64)
            steps = sigma[:, None] * f[f"{name}_scale"].astype(np.float64)
            mu = mu_t[f[f"{name}_ids"]].astype(np.float64)
            res = x.astype(np.float64) - mu
            for g in range(ng):
                sl = slice(g * G, (g + 1) * G)
                levels = steps[:, g, None, None] * (np.arange(4)[None, None, :] - f[f"{name}_zp"][:, g, None, None])
                dist = np.abs(res[:, sl, None] - levels)
                chosen = np.take_along_axis(dist, f[f"{name}_codes"][:, sl, None], axis=2)[..., 0]
                assert np.all(chosen <= dist.min(axis=2) + 1e-5 * steps[:, g, None] + 1e-30)
            # Eq. 2 step of each group (range extended to contain 0); a decoded step
            # below it can clip the group's ends by up to 3 |t - step|
            rg = res.reshape(len(res), ng, G)
            t = (np.maximum(rg.max(axis=2), 0) - np.minimum(rg.min(axis=2), 0)) / 3
            err = np.abs(xhat - x.astype(np.float64))
            bound = np.repeat(steps / 2 + 3 * np.abs(t - steps), G, axis=1) + 1e-6 * np.abs(x) + 1e-30
            assert np.all(err <= bound)


def test_append_gate_follows_the_keep_rule():
    # App. D.1 retention with the stored eigenvalues: a row is stored as written
    # without the gate exactly when the rule keeps it, else as zeros; with all
    # eigenvalues 0 every row is zeroed.
    import packed
    base = _small_workload(rank=4)
    gated = synth.scaled(base, storage=oracle.STORE_GATE)
    cfg0, tables, cache0, k, v, q, diag = _encoded(base)
    cfg1 = oracle.cfg_from_workload(gated)
    cache1 = oracle.new_cache(cfg1)
    oracle.append(cfg1, tables, cache1, 0, k, v)
    lay = packed.layout(base.batch, base.heads, base.head_dim, base.group_size, base.rank, base.capacity)
    kept = total = 0
    for h in range(base.heads):
        f0 = packed.fields(cache0, lay, h, 0, base.n_cache)
        f1 = packed.fields(cache1, lay, h, 0, base.n_cache)
        for t in range(base.n_cache):
            s0 = float(np.uint16(f0["k_cscale"][t]).view(np.float16))
            keep = oracle.keep_row(diag["coef"][0, h, t], f0["k_coef"][t], s0, tables[4][0, h])
            total += 1
            if keep:
                kept += 1
                np.testing.assert_array_equal(f1["k_coef"][t], f0["k_coef"][t])
                assert f1["k_cscale"][t] == f0["k_cscale"][t]
            else:
                assert not f1["k_coef"][t].any() and f1["k_cscale"][t] == 0
        for name in ("k_codes", "k_ids", "k_zp", "k_scale", "v_codes", "v_ids", "v_zp", "v_scale"):
            np.testing.assert_array_equal(f1[name], f0[name])
    assert kept > 0.9 * total
    zero_lam = tables[:4] + (np.zeros_like(tables[4]),)
    cache2 = oracle.new_cache(cfg1)
    oracle.append(cfg1, zero_lam, cache2, 0, k, v)
    for h in range(base.heads):
        f2 = packed.fields(cache2, lay, h, 0, base.n_cache)
        assert not f2["k_coef"].any() and not f2["k_cscale"].any()


# -------------------------------------- per-chunk coefficient layout (App. D.1)

def _read_coef_record(rec, n, r, nbh):
    """Reader of the chunk record format written from its definition: (layout,
    {(bh, t): (codes, scale bits)} of the stored rows, size)."""
    hdr = rec[:16].view("<u4")
    assert (int(hdr[1]), int(hdr[2]), int(hdr[3])) == (n, r, nbh)
    lay, rows = int(hdr[0]), {}
    if lay == oracle.COEF_DENSE:
        codes = rec[16:16 + nbh * n * r].reshape(nbh, n, r)
        scales = rec[16 + nbh * n * r:16 + nbh * n * (r + 2)].view("<u2").reshape(nbh, n)
        for bh in range(nbh):
            for t in range(n):
                rows[(bh, t)] = (codes[bh, t], int(scales[bh, t]))
        return lay, rows, 16 + nbh * n * (r + 2)
    assert lay == oracle.COEF_SPARSE
    counts = rec[16:16 + 4 * nbh].view("<u4")
    pos = 16 + 4 * nbh
    for bh in range(nbh):
        c = int(counts[bh])
        idx = rec[pos:pos + 2 * c].view("<u2")
        codes = rec[pos + 2 * c:pos + 2 * c + r * c].reshape(c, r)
        scales = rec[pos + 2 * c + r * c:pos + 4 * c + r * c].view("<u2")
        assert np.all(np.diff(idx.astype(np.int64)) > 0)
        for m in range(c):
            rows[(bh, int(idx[m]))] = (codes[m], int(scales[m]))
        pos += c * (r + 4)
    return lay, rows, pos


def _coef_cache(keep_frac, seed=31, rank=4):
    """An encoded cache whose coefficient rows outside a random keep set are
    zeroed, as the retention gate leaves them."""
    import packed
    wl = _small_workload(rank=rank)
    cfg, tables, cache, *_ = _encoded(wl)
    lay = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity)
    r = rng(seed)
    for bh in range(wl.batch * wl.heads):
        drop = np.nonzero(r.random(wl.n_cache) >= keep_frac)[0]
        packed.zero_coef_rows(cache, lay, bh, drop)
    return wl, cfg, cache, lay


@pytest.mark.parametrize("keep", [0.0, 0.1, 0.35, 0.7, 1.0])
def test_coef_record_round_trip(keep):
    # The record holds exactly the chunk's rows (all of them dense, the
    # non-zero-scale ones sparse, indices increasing); unpacking it into a
    # cache whose chunk rows hold garbage restores them and touches nothing else.
    import packed
    wl, cfg, cache, lay = _coef_cache(keep)
    start, n, nbh, r = 64, 130, wl.batch * wl.heads, wl.rank
    rec = oracle.coef_pack(cfg, cache, start, n)
    layout, rows, size = _read_coef_record(rec, n, r, nbh)
    assert size == rec.size
    for bh in range(nbh):
        f = packed.fields(cache, lay, bh, start, start + n)
        for t in range(n):
            kept = f["k_cscale"][t] != 0
            if layout == oracle.COEF_SPARSE and not kept:
                assert (bh, t) not in rows and not f["k_coef"][t].any()
                continue
            codes, sc = rows[(bh, t)]
            assert sc == f["k_cscale"][t] and np.array_equal(codes.view(np.int8), f["k_coef"][t])
    target = rng(5).integers(0, 256, cache.size, dtype=np.uint8)
    before = target.copy()
    oracle.coef_unpack(cfg, rec, target, start, n)
    chunk = packed.coef_byte_mask(lay, nbh, start, n)
    assert np.array_equal(target[chunk], cache[chunk])
    assert np.array_equal(target[~chunk], before[~chunk])


def test_coef_layout_choice_is_the_smaller_with_ties_dense():
    # Two heads, r = 4, a 4-token chunk: dense takes 16 + 2*4*6 = 64 bytes and
    # sparse 16 + 8 + 8k for k kept rows, so 5 kept rows tie (dense is kept) and
    # 4 go sparse; no kept row leaves only the counts.
    import packed
    wl, cfg, cache, lay = _coef_cache(1.0)
    start, n = 10, 4
    for k, want, size in [(8, oracle.COEF_DENSE, 64), (5, oracle.COEF_DENSE, 64), (4, oracle.COEF_SPARSE, 56),
                          (0, oracle.COEF_SPARSE, 24)]:
        c = cache.copy()
        drop = [(bh, t) for bh in range(2) for t in range(n)][k:]
        for bh, t in drop:
            packed.zero_coef_rows(c, lay, bh, [start + t])
        assert oracle.coef_record_bytes(cfg, c, start, n) == (size, want)
        assert oracle.coef_pack(cfg, c, start, n).size == size


def test_coef_record_of_a_fully_gated_chunk():
    # With all eigenvalues 0 the gate drops every row, and the record is the
    # header plus one zero count per head.
    wl = _small_workload(rank=4)
    gated = synth.scaled(wl, storage=oracle.STORE_GATE)
    cfg, tables, _, k, v, _, _ = _encoded(wl)
    cfg1 = oracle.cfg_from_workload(gated)
    cache = oracle.new_cache(cfg1)
    oracle.append(cfg1, tables[:4] + (np.zeros_like(tables[4]),), cache, 0, k, v)
    rec = oracle.coef_pack(cfg1, cache, 0, wl.n_cache)
    nbh = wl.batch * wl.heads
    assert rec.size == 16 + 4 * nbh and int(rec[:4].view("<u4")[0]) == oracle.COEF_SPARSE
    assert not rec[16:].any()


# ------------------------------------------------- BF16 active chunk (NEXT f2)

def test_active_chunk_alone_is_plain_attention():
    # Keys of the active chunk enter exactly, with no PSAC term: with an empty
    # packed history the oracle is torch's SDPA in fp64 on those Keys and Values,
    # under the block-causal mask over their positions.
    wl = _small_workload(rank=4)
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    n_act = wl.n_cache
    out, lse, _ = oracle.attend(cfg, tables, cache, 0, q, wl.q_start, wl.frame_tokens, k_act=k, v_act=v)
    for h in range(wl.heads):
        qh = q[0, :, h, :].astype(np.float64)
        ref = _sdpa(qh, k[0, :, h, :].astype(np.float64), v[0, :, h, :].astype(np.float64), _mask(wl, n_act))
        np.testing.assert_allclose(out[h * wl.n_q:(h + 1) * wl.n_q], ref, atol=1e-10)


def test_active_chunk_merges_by_log_sum_exp():
    # Softmax over disjoint key sets: attention over [packed | active] equals the
    # log-sum-exp merge of attention over each part (all keys visible here).
    wl = _small_workload(rank=4)
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    n_p, big = wl.n_cache - 100, 10 ** 6
    ka, va = np.ascontiguousarray(k[:, n_p:]), np.ascontiguousarray(v[:, n_p:])
    o_all, l_all, _ = oracle.attend(cfg, tables, cache, n_p, q, 0, big, k_act=ka, v_act=va)
    o_p, l_p, _ = oracle.attend(cfg, tables, cache, n_p, q, 0, big)
    o_a, l_a, _ = oracle.attend(cfg, tables, cache, 0, q, 0, big, k_act=ka, v_act=va)
    lse = np.logaddexp(l_p, l_a)
    ref = np.exp(l_p - lse)[:, None] * o_p + np.exp(l_a - lse)[:, None] * o_a
    np.testing.assert_allclose(l_all, lse, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(o_all, ref, atol=1e-12)


def test_active_chunk_empty_equals_packed_only():
    wl = _small_workload(rank=4)
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    e = np.zeros((1, 0, wl.heads, wl.head_dim), np.float32)
    a = oracle.attend(cfg, tables, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens, k_act=e, v_act=e)
    b = oracle.attend(cfg, tables, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])


# ------------------------------------------- per-chunk calibration epochs (NEXT f1)

def _two_epoch_cache(wl):
    """Chunk 1 appended with tables calibrated on it, chunk 2 with tables
    recalibrated on chunk 2 (and a second, different Query history)."""
    cfg = oracle.cfg_from_workload(wl)
    k = synth.tensor(wl, "k", wl.n_cache)
    v = synth.tensor(wl, "v", wl.n_cache)
    qh = synth.tensor(wl, "qhist", 2 * wl.n_hist)
    split = wl.n_cache // 2 + 7
    t1 = oracle.calibrate(cfg, qh[:, :wl.n_hist], k[:, :split], v[:, :split], 5)
    t2 = oracle.calibrate(cfg, qh, k[:, split:], v[:, split:], 5)
    cache = oracle.new_cache(cfg)
    oracle.append(cfg, t1, cache, 0, np.ascontiguousarray(k[:, :split]), np.ascontiguousarray(v[:, :split]))
    oracle.append(cfg, t2, cache, split, np.ascontiguousarray(k[:, split:]), np.ascontiguousarray(v[:, split:]))
    return cfg, k, v, split, t1, t2, cache


def test_single_epoch_equals_plain_attention():
    wl = _small_workload(rank=4)
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    a = oracle.attend(cfg, tables, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    b = oracle.attend(cfg, None, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens, epochs=[(0, tables)])
    np.testing.assert_array_equal(a[0], b[0])
    c = oracle.attend(cfg, None, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens,
                      epochs=[(0, tables), (77, tables), (150, tables)])
    np.testing.assert_array_equal(a[0], c[0])
    np.testing.assert_array_equal(a[1], c[1])


def test_epochs_match_explicit_reconstruction_fp32():
    # Each key decodes with its epoch's centroids, and its Eq. 17 term uses its
    # epoch's U_r: attention equals torch's SDPA (fp64) over the explicitly
    # reconstructed Khat = Khat_0 + chat U_r^(e)T, epoch by epoch.
    wl = _small_workload(rank=4)
    cfg, k, v, split, t1, t2, cache = _two_epoch_cache(wl)
    q = synth.tensor(wl, "q", wl.n_q)
    out, _, _ = oracle.attend(cfg, None, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens,
                              epochs=[(0, t1), (split, t2)])
    plain, _, _ = oracle.attend(cfg, t1, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    for h in range(wl.heads):
        rows_k, rows_v = [], []
        for (s0, s1, t) in ((0, split, t1), (split, wl.n_cache, t2)):
            k0, ch, vh = oracle.decode(cfg, t, cache, 0, h, wl.n_cache)
            rows_k.append(k0[s0:s1] + ch[s0:s1] @ t[3][0, h].astype(np.float64))
            rows_v.append(vh[s0:s1])
        Khat, Vhat = np.concatenate(rows_k), np.concatenate(rows_v)
        ref = _sdpa(q[0, :, h, :].astype(np.float64), Khat, Vhat, _mask(wl, wl.n_cache))
        got = out[h * wl.n_q:(h + 1) * wl.n_q]
        assert np.abs(got - ref).max() < 1e-5
        # and decoding the second chunk with the first epoch's tables is wrong
        assert np.abs(plain[h * wl.n_q:(h + 1) * wl.n_q] - ref).max() > 1e-3


# ------------------------------------- INT8 PSAC rows (App. D.1, Eq. 16)

def _f16(x):
    """IEEE binary16 round-to-nearest-even of an fp32 value (numpy's cast), as a float."""
    return float(np.float32(np.float16(np.float32(x))))


def _row_rule(C):
    """The App. D.1 row written from its statement (reading R10): s = RN16(max|C| / 127),
    saturating at the largest binary16; codes RN(C / s) clamped to +-127; 0 when s = 0."""
    C = np.asarray(C, np.float32)
    amax = np.float32(np.abs(C).max()) if C.size else np.float32(0)
    s = np.float32(min(np.float32(amax / np.float32(127.0)), np.float32(65504.0)))
    s = np.float32(_f16(s))
    if s == 0:
        return np.zeros(C.size, np.int8), s
    return np.clip(np.rint(C / s), -127, 127).astype(np.int8), s


def test_coef_row_hand_examples():
    # scale 2^-7 exactly (0.9921875 / 127); 2.5 and -2.5 steps round to even, 3.5 up
    s = 2.0 ** -7
    codes, sb = oracle.coef_row([127 * s, 2.5 * s, 3.5 * s, -2.5 * s, 0.0, -127 * s])
    assert list(codes) == [127, 2, 4, -2, 0, -127]
    assert sb == 0x2000  # binary16 2^-7
    # a zero row stores zero codes and a zero scale
    codes, sb = oracle.coef_row([0.0, 0.0, 0.0])
    assert not codes.any() and sb == 0
    # a scale below half the smallest binary16 subnormal rounds to 0: the row is zero
    codes, sb = oracle.coef_row([1e-6, -5e-7])
    assert not codes.any() and sb == 0
    # saturation: max|C| / 127 above 65504 stores 65504 (0x7bff) and clamps the codes
    codes, sb = oracle.coef_row([1e7, 3 * 65504.0, -1e7, 0.4 * 65504.0])
    assert sb == 0x7BFF and list(codes) == [127, 3, -127, 0]
    # the largest element lands on +-127 up to the scale's binary16 rounding
    codes, sb = oracle.coef_row([0.3, -1.0, 0.05])
    s16 = oracle.f16_value(sb)
    assert s16 == _f16(1.0 / 127.0) and codes[1] == -127 and codes[0] == round(0.3 / s16)


def test_coef_row_matches_the_rule_and_error_bound():
    r = rng(31)
    for n in range(600):
        rank = int(r.integers(1, 33))
        mag = 10.0 ** r.uniform(-6, 6)
        C = (r.standard_normal(rank) * mag).astype(np.float32)
        if n % 7 == 0:
            C[r.integers(rank)] = 0.0
        codes, sb = oracle.coef_row(C)
        want, s = _row_rule(C)
        np.testing.assert_array_equal(codes, want)
        assert oracle.f16_value(sb) == float(s)
        if s > 0:
            inside = np.abs(C / s) <= 127.0
            err = np.abs(C.astype(np.float64) - codes.astype(np.float64) * float(s))
            assert np.all(err[inside] <= float(s) / 2 * (1 + 1e-6))


def test_append_stores_int8_rows_of_its_coefficients():
    # The cache's INT8 rows and FP16 row scales are the App. D.1 encoding of the
    # fp32 coefficients C = (k - khat_0) U_r that append computed.
    from packed import fields, layout
    for dt in ("f32", "bf16"):
        wl = _small_workload(rank=12, head_dim=32, group_size=16, dtype=dt)
        cfg, tables, cache, k, v, q, diag = _encoded(wl)
        lay = layout(1, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity)
        nz = 0
        for h in range(wl.heads):
            f = fields(cache, lay, h, 0, wl.n_cache)
            for t in range(wl.n_cache):
                C = diag["coef"][0, h, t]
                want, s = _row_rule(C)
                np.testing.assert_array_equal(f["k_coef"][t], want)
                assert oracle.f16_value(int(f["k_cscale"][t])) == float(s)
                nz += int(s > 0)
        assert nz > wl.heads * wl.n_cache // 2


# -------------------------------- BF16 operands of Eq. 17 attention (reading R15)

def _bf16_f64(x):
    """Round float64 values to BF16 (8 significant bits) once, ties to even, by
    truncating the binary64 significand with a rounding bias."""
    x = np.ascontiguousarray(x, np.float64)
    bits = x.view(np.uint64)
    lsb = (bits >> np.uint64(45)) & np.uint64(1)
    out = (bits + np.uint64((1 << 44) - 1) + lsb) & ~np.uint64((1 << 45) - 1)
    return out.view(np.float64)


def _sdpa_aug(q, u, K, C, V, mask, d):
    """fp64 SDPA over the augmented depth d + r: ([q | u] . [K | C]) / sqrt(d)."""
    qa = np.concatenate([q, u], 1)
    ka = np.concatenate([K, C], 1)
    qt = torch.from_numpy(qa)[None]
    return torch.nn.functional.scaled_dot_product_attention(
        qt, torch.from_numpy(ka)[None], torch.from_numpy(V)[None], attn_mask=torch.from_numpy(mask)[None],
        scale=1.0 / math.sqrt(d))[0].numpy()


def _bf16_reference(wl, cfg, tables, cache, q, h, n_cache, rounded=True):
    k0, ch, vh = oracle.decode(cfg, tables, cache, 0, h, n_cache)
    U = tables[3][0, h].astype(np.float64)  # [r, d], BF16 values
    qh = q[0, :, h, :].astype(np.float64)
    u = qh @ U.T
    if rounded:
        k0, ch, vh, u = _bf16_f64(k0), _bf16_f64(ch), _bf16_f64(vh), _bf16_f64(u)
    return qh, u, k0, ch, vh


def test_attend_bf16_operands_are_rounded():
    # BF16 workloads (App. D.1 keeps centroids and U_r in BF16 and attends over
    # BF16 K/V): the oracle's Eq. 17 logits take khat_0, vhat, chat and q U_r
    # rounded to BF16. Reference: fp64 SDPA over those operands rounded here
    # independently; the same reference without the rounding is measurably off.
    wl = _small_workload(rank=4, dtype="bf16")
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    out, lse, _ = oracle.attend(cfg, tables, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    mask = _mask(wl, wl.n_cache)
    for h in range(wl.heads):
        got = out[h * wl.n_q:(h + 1) * wl.n_q]
        qh, u, k0, ch, vh = _bf16_reference(wl, cfg, tables, cache, q, h, wl.n_cache)
        ref = _sdpa_aug(qh, u, k0, ch, vh, mask, wl.head_dim)
        assert np.abs(got - ref).max() < 1e-10
        qh, u, k0, ch, vh = _bf16_reference(wl, cfg, tables, cache, q, h, wl.n_cache, rounded=False)
        loose = _sdpa_aug(qh, u, k0, ch, vh, mask, wl.head_dim)
        assert np.abs(got - loose).max() > 1e-4
        # each rounding point on its own matters
        qh, u, k0, ch, vh = _bf16_reference(wl, cfg, tables, cache, q, h, wl.n_cache)
        u_raw = q[0, :, h, :].astype(np.float64) @ tables[3][0, h].astype(np.float64).T
        assert np.abs(got - _sdpa_aug(qh, u_raw, k0, ch, vh, mask, wl.head_dim)).max() > 1e-7
        k0_raw, _, v_raw = oracle.decode(cfg, tables, cache, 0, h, wl.n_cache)
        assert np.abs(got - _sdpa_aug(qh, u, k0_raw, ch, vh, mask, wl.head_dim)).max() > 1e-5
        assert np.abs(got - _sdpa_aug(qh, u, k0, ch, v_raw, mask, wl.head_dim)).max() > 1e-5


def test_active_chunk_bf16_matches_rounded_reference():
    # [packed | active] in BF16: the packed keys as above, the active chunk's exact
    # tokens (BF16 already) with no PSAC term.
    wl = _small_workload(rank=4, dtype="bf16")
    cfg, tables, cache, k, v, q, _ = _encoded(wl)
    n_p = wl.n_cache - 90
    ka, va = np.ascontiguousarray(k[:, n_p:]), np.ascontiguousarray(v[:, n_p:])
    out, _, _ = oracle.attend(cfg, tables, cache, n_p, q, wl.q_start, wl.frame_tokens, k_act=ka, v_act=va)
    mask = _mask(wl, wl.n_cache)
    for h in range(wl.heads):
        qh, u, k0, ch, vh = _bf16_reference(wl, cfg, tables, cache, q, h, n_p)
        K = np.concatenate([k0, _bf16_f64(ka[0, :, h].astype(np.float64))])
        C = np.concatenate([ch, np.zeros((wl.n_cache - n_p, wl.rank))])
        V = np.concatenate([vh, _bf16_f64(va[0, :, h].astype(np.float64))])
        ref = _sdpa_aug(qh, u, K, C, V, mask, wl.head_dim)
        assert np.abs(out[h * wl.n_q:(h + 1) * wl.n_q] - ref).max() < 1e-10


def test_epochs_bf16_match_rounded_reference():
    # Two calibration epochs in BF16: every key decodes with its epoch's centroids
    # and pairs its chat with q U_r of its epoch, all operands rounded to BF16.
    wl = _small_workload(rank=4, dtype="bf16")
    cfg, k, v, split, t1, t2, cache = _two_epoch_cache(wl)
    q = synth.tensor(wl, "q", wl.n_q)
    out, _, _ = oracle.attend(cfg, None, cache, wl.n_cache, q, wl.q_start, wl.frame_tokens,
                              epochs=[(0, t1), (split, t2)])
    mask = _mask(wl, wl.n_cache)
    for h in range(wl.heads):
        parts = []
        for (s0, s1, t) in ((0, split, t1), (split, wl.n_cache, t2)):
            qh, u, k0, ch, vh = _bf16_reference(wl, cfg, t, cache, q, h, wl.n_cache)
            parts.append((u, k0[s0:s1], ch[s0:s1], vh[s0:s1]))
        # logits by hand: each epoch's keys with that epoch's u
        L = np.concatenate([(qh @ K0.T + u @ C.T) for (u, K0, C, _) in parts], 1) / math.sqrt(wl.head_dim)
        V = np.concatenate([p[3] for p in parts])
        L = np.where(mask, L, -np.inf)
        P = np.exp(L - L.max(1, keepdims=True))
        ref = (P @ V) / P.sum(1, keepdims=True)
        assert np.abs(out[h * wl.n_q:(h + 1) * wl.n_q] - ref).max() < 1e-10


# ------------------------------------- K-means with an empty cluster (Eq. 3, R1)

def _lloyd_reference(x, kc, iters, table):
    """Lloyd written from reading R1: initial centroids are tokens floor(j n / Kc);
    assignment by fp32 squared distance summed over channels in order, ties to the
    lower index; the update is the fp64 token-order mean rounded to the table type;
    a cluster with no token keeps its centroid."""
    n, d = x.shape
    rnd = (lambda a: np.asarray(a, np.float32)) if table == "f32" else (lambda a: _bf16_f64(a).astype(np.float32))
    mu = rnd(x[[(j * n) // kc for j in range(kc)]].astype(np.float64))
    empty = 0
    for _ in range(iters):
        acc = np.zeros((n, kc), np.float32)
        for c in range(d):
            t = (x[:, None, c] - mu[None, :, c]).astype(np.float32)
            acc = (acc + t * t).astype(np.float32)
        assign = np.argmin(acc, 1)  # first minimum: the lower index
        sums = np.zeros((kc, d))
        counts = np.zeros(kc, np.int64)
        for t_ in range(n):
            sums[assign[t_]] += x[t_].astype(np.float64)
            counts[assign[t_]] += 1
        for j in range(kc):
            if counts[j] > 0:
                mu[j] = rnd(sums[j] / counts[j])
            else:
                empty += 1
    return mu, empty


@pytest.mark.parametrize("dt", ["f32", "bf16"])
def test_kmeans_empty_cluster_keeps_its_centroid(dt):
    # Tokens 0 and 10 (the initial picks of clusters 0 and 1) are equal, so the
    # two starting centroids coincide and every tie goes to cluster 0: cluster 1
    # is empty in the first iteration and must keep its initial centroid. Later
    # iterations (cluster 0 has moved) follow the reference bit for bit.
    r = rng(41)
    d, kc, n = 16, 4, 40
    x = (r.standard_normal((n, d)) * 3).astype(np.float32)
    x = synth.round_to(x, dt)
    x[10] = x[0]
    wl = _small_workload(head_dim=d, n_centroids=kc, group_size=16, rank=0, heads=1, dtype=dt)
    cfg = oracle.cfg_from_workload(wl)
    xt = np.ascontiguousarray(x[None, :, None, :])
    mu1, _, _, _, _ = oracle.calibrate(cfg, None, xt, xt, 1)
    ref1, empty1 = _lloyd_reference(x, kc, 1, dt)
    assert empty1 == 1
    np.testing.assert_array_equal(mu1[0, 0], ref1)
    np.testing.assert_array_equal(mu1[0, 0, 1], x[10])
    mu6, _, _, _, _ = oracle.calibrate(cfg, None, xt, xt, 6)
    ref6, _ = _lloyd_reference(x, kc, 6, dt)
    np.testing.assert_array_equal(mu6[0, 0], ref6)


def test_kmeans_matches_reference_lloyd_on_overlapping_data():
    # Overlapping clusters (assignments change between iterations), against the
    # same reference Lloyd, bit for bit.
    r = rng(42)
    d, kc, n = 8, 6, 300
    x = (r.standard_normal((n, d)) + r.integers(0, 3, size=(n, 1))).astype(np.float32)
    wl = _small_workload(head_dim=d, n_centroids=kc, group_size=8, rank=0, heads=1)
    cfg = oracle.cfg_from_workload(wl)
    xt = np.ascontiguousarray(x[None, :, None, :])
    mu_k, _, _, _, _ = oracle.calibrate(cfg, None, xt, xt, 7)
    ref, _ = _lloyd_reference(x, kc, 7, "f32")
    np.testing.assert_array_equal(mu_k[0, 0], ref)


# ---------------------------------------------------------- oracle bounds

def test_oracle_rejects_head_dim_above_256():
    # The oracle's per-token buffers hold 256 channels: larger head_dim is refused.
    cfg = oracle.cfg_of(1, 1, 512, 4, 32, 4, 2, 64, False)
    assert oracle.cache_bytes(cfg) == -1
    x = np.zeros((1, 8, 1, 512), np.float32)
    with pytest.raises(RuntimeError):
        oracle.calibrate(cfg, None, x, x, 1)
    ok = oracle.cfg_of(1, 1, 256, 4, 32, 4, 2, 64, False)
    assert oracle.cache_bytes(ok) > 0


# ---------------------------- resident sparse PSAC rows (App. D.1, reading R26)

def _planted(wl, drop, seed=3):
    """Inputs whose tokens in `drop` (a set of positions) equal a centroid of
    their head exactly: a zero residual, so E = 0, C = 0 and a zero row (App.
    D.1 drops it). Calibration uses the unplanted first chunk."""
    cfg0 = oracle.cfg_from_workload(synth.scaled(wl, storage=wl.storage & ~oracle.STORE_SPARSE, coef_rows=0))
    k = synth.tensor(wl, "k", wl.n_cache)
    v = synth.tensor(wl, "v", wl.n_cache)
    qh = synth.tensor(wl, "qhist", wl.n_hist)
    tables = oracle.calibrate(cfg0, qh, k[:, :wl.chunk], v[:, :wl.chunk], 5)
    r = rng(seed)
    for b in range(wl.batch):
        for h in range(wl.heads):
            for t in sorted(drop):
                k[b, t, h] = tables[0][b, h, r.integers(wl.n_centroids)]
    return k, v, tables


def _append_chunks(cfg, tables, k, v, chunks):
    cache = oracle.new_cache(cfg)
    for s0, n in chunks:
        oracle.append(cfg, tables, cache, s0, np.ascontiguousarray(k[:, s0:s0 + n]),
                      np.ascontiguousarray(v[:, s0:s0 + n]))
    return cache


def _sparse_wl(**kw):
    base = dict(rank=12, head_dim=32, group_size=16, n_cache=900, n_q=96, q_start=804, frame_tokens=32,
                chunk=300, storage=oracle.STORE_GATE | oracle.STORE_SPARSE, heads=2, batch=2)
    base.update(kw)
    return _small_workload(**base)


# chunk 0 drops nothing, chunk 1 drops two rows (still dense: 2 x 14 B < 38 B of
# mask), chunk 2 drops 40% of its rows (sparse); chunk boundaries inside tiles
_CHUNKS = [(0, 300), (300, 300), (600, 300)]
_DROP = {310, 451} | set(range(600, 900, 5)) | set(range(601, 900, 5))


def test_sparse_rows_decode_like_the_gated_dense_cache():
    wl = _sparse_wl()
    k, v, tables = _planted(wl, _DROP)
    dense = synth.scaled(wl, storage=oracle.STORE_GATE)
    cs = _append_chunks(oracle.cfg_from_workload(wl), tables, k, v, _CHUNKS)
    cd = _append_chunks(oracle.cfg_from_workload(dense), tables, k, v, _CHUNKS)
    cfg_s, cfg_d = oracle.cfg_from_workload(wl), oracle.cfg_from_workload(dense)
    for b in range(wl.batch):
        for h in range(wl.heads):
            a = oracle.decode(cfg_s, tables, cs, b, h, wl.n_cache)
            c = oracle.decode(cfg_d, tables, cd, b, h, wl.n_cache)
            for x, y in zip(a, c):
                np.testing.assert_array_equal(x, y)
            assert not a[1][sorted(_DROP)].any()
    q = synth.tensor(wl, "q", wl.n_q)
    o1 = oracle.attend(cfg_s, tables, cs, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    o2 = oracle.attend(cfg_d, tables, cd, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    np.testing.assert_array_equal(o1[0], o2[0])
    np.testing.assert_array_equal(o1[1], o2[1])


def test_sparse_directory_and_pool_follow_the_chunk_rule():
    # Read with an independent reader of the documented layout: each chunk is
    # stored dense (all rows) or sparse (non-zero-scale rows only), whichever is
    # smaller with one mask bit per slot; rows in slot order; bases are prefix
    # counts; the pool rows are the rows the gated dense cache holds.
    import packed
    wl = _sparse_wl()
    k, v, tables = _planted(wl, _DROP)
    cs = _append_chunks(oracle.cfg_from_workload(wl), tables, k, v, _CHUNKS)
    dense = synth.scaled(wl, storage=oracle.STORE_GATE)
    cd = _append_chunks(oracle.cfg_from_workload(dense), tables, k, v, _CHUNKS)
    ls = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity, wl.storage, 0,
                       wl.chunk)
    ld = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity, dense.storage)
    r = wl.rank
    modes = []
    for bh in range(wl.batch * wl.heads):
        fd = packed.fields(cd, ld, bh, 0, wl.n_cache)
        base, mask = packed.directory(cs, ls, bh)
        codes, scale = packed.pool(cs, ls, bh)
        stored = np.zeros(wl.n_cache, bool)
        for s0, n in _CHUNKS:
            kept = int((fd["k_cscale"][s0:s0 + n] != 0).sum())
            sparse = kept * (r + 2) + (n + 7) // 8 < n * (r + 2)
            modes.append(sparse)
            stored[s0:s0 + n] = (fd["k_cscale"][s0:s0 + n] != 0) if sparse else True
        rows = np.cumsum(stored) - 1
        for t in range(wl.n_cache):
            T, i = divmod(t, 64)
            assert bool((int(mask[T]) >> i) & 1) == stored[t]
            if i == 0:
                assert base[T] == stored[:t].sum()
            if stored[t]:
                np.testing.assert_array_equal(codes[rows[t]], fd["k_coef"][t])
                assert scale[rows[t]] == fd["k_cscale"][t]
        assert packed.overflow(cs, ls, bh) == 0
        print(f"head {bh}: {stored.sum()} pool rows for {wl.n_cache} slots")
    assert modes[:3] == [False, False, True]


def test_sparse_pool_overflow_drops_and_counts_rows():
    # A pool of 700 rows for 900 slots holding more: the rows past its end are not
    # stored and are counted; they read as zero rows, so attention equals the
    # gated dense cache with exactly those rows zeroed.
    import packed
    wl = _sparse_wl(coef_rows=700)
    k, v, tables = _planted(wl, _DROP)
    cfg_s = oracle.cfg_from_workload(wl)
    cs = _append_chunks(cfg_s, tables, k, v, _CHUNKS)
    dense = synth.scaled(wl, storage=oracle.STORE_GATE, coef_rows=0)
    cfg_d = oracle.cfg_from_workload(dense)
    cd = _append_chunks(cfg_d, tables, k, v, _CHUNKS)
    ls = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity, wl.storage, 700,
                       wl.chunk)
    ld = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity, dense.storage)
    for bh in range(wl.batch * wl.heads):
        b, h = divmod(bh, wl.heads)
        _, ch_s, _ = oracle.decode(cfg_s, tables, cs, b, h, wl.n_cache)
        _, ch_d, _ = oracle.decode(cfg_d, tables, cd, b, h, wl.n_cache)
        lost = np.nonzero(np.abs(ch_d).sum(1) != np.abs(ch_s).sum(1))[0]
        assert len(lost) == packed.overflow(cs, ls, bh) > 0
        assert not ch_s[lost].any() and lost.min() >= 600  # only the last chunk spills
        packed.zero_coef_rows(cd, ld, bh, lost)
    q = synth.tensor(wl, "q", wl.n_q)
    o1 = oracle.attend(cfg_s, tables, cs, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    o2 = oracle.attend(cfg_d, tables, cd, wl.n_cache, q, wl.q_start, wl.frame_tokens)
    np.testing.assert_array_equal(o1[0], o2[0])


def test_sparse_reappend_over_the_same_slots_is_idempotent():
    # Appending a chunk again into the same slots (rows in slot order, the fill
    # read from the directory below the chunk) leaves the cache unchanged.
    wl = _sparse_wl()
    k, v, tables = _planted(wl, _DROP)
    cfg = oracle.cfg_from_workload(wl)
    cs = _append_chunks(cfg, tables, k, v, _CHUNKS)
    again = cs.copy()
    for s0, n in _CHUNKS[1:]:
        oracle.append(cfg, tables, again, s0, np.ascontiguousarray(k[:, s0:s0 + n]),
                      np.ascontiguousarray(v[:, s0:s0 + n]))
    over_lay = __import__("packed").layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity,
                                           wl.storage, 0, wl.chunk)
    np.testing.assert_array_equal(cs, again)
    assert over_lay["total"] == cs.size


def test_sparse_cache_bytes():
    import packed
    for rows in (0, 640, 1000):
        wl = _sparse_wl(coef_rows=rows)
        cfg = oracle.cfg_from_workload(wl)
        lay = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.capacity, wl.storage, rows,
                            wl.chunk)
        assert oracle.cache_bytes(cfg) == lay["total"]
    # an append of more tokens than the staging rows hold is refused
    wl = _sparse_wl()
    k, v, tables = _planted(wl, set())
    with pytest.raises(RuntimeError):
        oracle.append(oracle.cfg_from_workload(wl), tables, oracle.new_cache(oracle.cfg_from_workload(wl)), 0,
                      np.ascontiguousarray(k[:, :wl.chunk + 1]), np.ascontiguousarray(v[:, :wl.chunk + 1]))
    # sparse rows need r >= 1
    assert oracle.cache_bytes(oracle.cfg_from_workload(_sparse_wl(rank=0))) == -1
    # the chunk records read slot-addressed rows: refused on a sparse cache
    wl = _sparse_wl()
    with pytest.raises(RuntimeError):
        oracle.coef_pack(oracle.cfg_from_workload(wl), oracle.new_cache(oracle.cfg_from_workload(wl)), 0, 10)
