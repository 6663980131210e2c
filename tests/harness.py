"""Builds parity cases: seeded inputs, the oracle's results on a set of source
heads, and full-size GPU launches whose heads replicate those sources.

At the full sizes of the benchmark workloads the oracle cannot afford every
head, so it computes a few source heads and every head of the GPU launch
carries the inputs of one source (round-robin). The GPU then runs in exactly
the launch configuration that bench.py times, and every GPU head is compared
with the oracle's result for its source.
"""
from __future__ import annotations

import dataclasses
import math

import numpy as np

import oracle
import synth
import packed


@dataclasses.dataclass
class OracleCase:
    wl: synth.Workload
    sources: list            # [(b, h)] of the generator, in source order
    src_of: np.ndarray       # [B * H] -> source index
    k: np.ndarray            # [1, n_cache, S, d] float32 source inputs
    v: np.ndarray
    q: np.ndarray            # [1, n_q, S, d]
    tables: tuple            # (mu_k, mu_v, w, u_t, lam), each [1, S, ...]
    cfg: object              # oracle config of the sources (B = 1, H = S)
    cache: np.ndarray        # oracle cache of the sources
    diag: dict               # oracle append diagnostics
    lay: dict                # packed layout of the source cache


def sources_for(wl: synth.Workload, max_sources: int):
    allh = [(b, h) for b in range(wl.batch) for h in range(wl.heads)]
    if len(allh) <= max_sources:
        return allh
    pick = np.linspace(0, len(allh) - 1, max_sources).round().astype(int)
    return [allh[i] for i in sorted(set(pick.tolist()))]


def _gen_sources(wl, sources, what, n):
    out = np.zeros((1, n, len(sources), wl.head_dim), np.float32)
    fn = {"k": synth.keys_head, "v": synth.values_head,
          "q": lambda w, b, h, m: synth.queries_head(w, b, h, m, False),
          "qhist": lambda w, b, h, m: synth.queries_head(w, b, h, m, True)}[what]
    for s, (b, h) in enumerate(sources):
        out[0, :, s, :] = synth.round_to(fn(wl, b, h, n), wl.dtype)
    return out


def build_oracle_case(wl: synth.Workload, max_sources: int = 3, cold: bool = False, transform=None,
                      tables_edit=None) -> OracleCase:
    """transform(k, v, q) -> (k, v, q) edits the generated source inputs (for edge
    cases); its results are rounded to the workload's dtype. tables_edit(tables)
    edits the calibrated tables in place before the cache is appended."""
    sources = sources_for(wl, max_sources)
    S = len(sources)
    cfg = oracle.cfg_of(1, S, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank, wl.top_m,
                        wl.n_cache, wl.dtype == "bf16", wl.storage, wl.metric)
    k = _gen_sources(wl, sources, "k", wl.n_cache)
    v = _gen_sources(wl, sources, "v", wl.n_cache)
    q = _gen_sources(wl, sources, "q", wl.n_q)
    if transform is not None:
        k, v, q = (np.ascontiguousarray(synth.round_to(np.asarray(x, np.float32), wl.dtype))
                   for x in transform(k, v, q))
    qh = None if cold else _gen_sources(wl, sources, "qhist", wl.n_hist)
    nc = min(wl.chunk, wl.n_cache)
    tables = oracle.calibrate(cfg, qh, np.ascontiguousarray(k[:, :nc]), np.ascontiguousarray(v[:, :nc]),
                              wl.kmeans_iters)
    if tables_edit is not None:
        tables_edit(tables)
    cache = oracle.new_cache(cfg)
    diag = oracle.append(cfg, tables, cache, 0, k, v, diagnostics=True)
    lay = packed.layout(1, S, wl.head_dim, wl.group_size, wl.rank, wl.n_cache, wl.storage, wl.coef_rows,
                         wl.coef_stage or wl.chunk)
    bh = wl.batch * wl.heads
    src_of = np.arange(bh) % S
    if S == bh:
        src_of = np.arange(bh)
    return OracleCase(wl, sources, src_of, k, v, q, tables, cfg, cache, diag, lay)


def full_inputs(case: OracleCase, what: str) -> np.ndarray:
    """[B, n, H, d] float32: every head carries its source's tokens."""
    wl = case.wl
    src = {"k": case.k, "v": case.v, "q": case.q}[what]
    n = src.shape[1]
    out = np.empty((wl.batch, n, wl.heads, wl.head_dim), np.float32)
    for bh in range(wl.batch * wl.heads):
        b, h = divmod(bh, wl.heads)
        out[b, :, h, :] = src[0, :, case.src_of[bh], :]
    return out


def full_tables(case: OracleCase):
    wl = case.wl
    out = []
    for t in case.tables:
        rep = t[0][case.src_of]  # [B*H, ...]
        out.append(np.ascontiguousarray(rep.reshape((wl.batch, wl.heads) + t.shape[2:])))
    return out


def full_oracle_cache(case: OracleCase) -> np.ndarray:
    wl = case.wl
    lay = packed.layout(wl.batch, wl.heads, wl.head_dim, wl.group_size, wl.rank, wl.n_cache, wl.storage,
                         wl.coef_rows, wl.coef_stage or wl.chunk)
    out = np.zeros(lay["total"], np.uint8)
    for bh in range(wl.batch * wl.heads):
        packed.copy_head(out, lay, bh, case.cache, case.lay, int(case.src_of[bh]), wl.n_cache)
    return out


def sample_rows(wl: synth.Workload, n_heads_max: int, step: int, src_of=None):
    """(b, h, i) rows of the full launch: a spread of heads, every step-th Query."""
    bh_all = np.arange(wl.batch * wl.heads)
    pick = bh_all if len(bh_all) <= n_heads_max else \
        np.unique(np.linspace(0, len(bh_all) - 1, n_heads_max).round().astype(int))
    idx = np.unique(np.concatenate([np.arange(0, wl.n_q, step), [wl.n_q - 1]]))
    rows = [(bh // wl.heads, bh % wl.heads, i) for bh in pick for i in idx]
    return np.array(rows, np.int32)


# ------------------------------------------------------------ near ties

def qsac_near_tie(k, mu, w, M, rel=2.0 ** -16):
    """True if the fp64 Eq. 9 distances put the M-th and (M+1)-th centroid within
    the fp32 rounding of the two distance forms (expanded on the GPU, literal in
    the oracle); such a token may legitimately pick another candidate set."""
    k = k.astype(np.float64); mu = mu.astype(np.float64); w = w.astype(np.float64)
    dq = ((k[None, :] - mu) ** 2 * w[None, :]).sum(1)
    mag = (w[None, :] * (k[None, :] ** 2 + mu ** 2)).sum(1)
    o = np.argsort(dq, kind="stable")
    if M >= len(dq):
        return False
    a, b = o[M - 1], o[M]
    return abs(dq[b] - dq[a]) <= rel * (mag[a] + mag[b])


def qsac_near_tie_full(k, mu, m, M, rel=2.0 ** -16):
    """The same for the full quadratic form (k - mu)^T m (k - mu): the GPU ranks
    with the expanded constants m mu_j, the oracle with the literal form; both
    round within rel times (|k| + |mu|)^T |m| (|k| + |mu|)."""
    k = k.astype(np.float64); mu = mu.astype(np.float64); m = m.astype(np.float64)
    e = k[None, :] - mu
    dq = np.einsum("jc,cd,jd->j", e, m, e)
    a = np.abs(k)[None, :] + np.abs(mu)
    mag = np.einsum("jc,cd,jd->j", a, np.abs(m), a)
    o = np.argsort(dq, kind="stable")
    if M >= len(dq):
        return False
    i, j = o[M - 1], o[M]
    return abs(dq[j] - dq[i]) <= rel * (mag[i] + mag[j])


def nearest_near_tie(x, mu, rel=2.0 ** -16):
    x = x.astype(np.float64); mu = mu.astype(np.float64)
    dd = ((x[None, :] - mu) ** 2).sum(1)
    mag = (x[None, :] ** 2 + mu ** 2).sum(1)
    o = np.argsort(dd, kind="stable")
    if len(dd) < 2:
        return False
    a, b = o[0], o[1]
    return abs(dd[b] - dd[a]) <= rel * (mag[a] + mag[b])


def near_half(x, tol=1e-4):
    f = np.abs(x - np.floor(x) - 0.5)
    return f <= tol


def f16_boundary(x, rel=1e-5):
    """True where x lies within rel of a midpoint between two binary16 values."""
    x = np.abs(np.asarray(x, np.float64))
    lo = x.astype(np.float16).astype(np.float64)
    nxt = np.nextafter(x.astype(np.float16), np.float16(np.inf)).astype(np.float64)
    prv = np.nextafter(x.astype(np.float16), np.float16(0)).astype(np.float64)
    mids = np.stack([(lo + nxt) / 2, (lo + prv) / 2], -1)
    return (np.abs(mids - x[..., None]) <= rel * np.maximum(x[..., None], 1e-30)).any(-1)


def rel_inf(a, b):
    return float(np.max(np.abs(a - b))) / max(float(np.max(np.abs(b))), 1e-30)


def lse_tol(lse):
    return 1e-3 * (1.0 + np.abs(lse))


def isqrt(d):
    return 1.0 / math.sqrt(d)
