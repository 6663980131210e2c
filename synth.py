"""Seeded synthetic workloads shaped like the attention of causal video world models.

This module only draws inputs. It holds none of QuantWM's arithmetic, so both
the CPU oracle (``oracle/``) and the HIP path consume exactly the same tensors.

Input recipe, per (batch b, head h). Every stream is a Philox4x32 counter-based
generator (Salmon et al., SC'11, as shipped by numpy) keyed on
``(seed, b, h, stream)``, so any head can be regenerated alone:

* Keys: channel std ``sigma_c = exp(N(0,1))`` (LogNormal(0,1)); ``n_out``
  distinct outlier channels (seeded permutation) get ``sigma_c *= out_scale``;
  16 mixture means ``m_k = sigma * N(0, I)``; each token draws a uniform label k
  and is ``m_k + 0.5 * sigma * N(0, I)``.
* Values: ``N(0, I)``.
* Queries (the chunk and the historical stream): ``N(0, I) + 5 * A u`` with
  ``u ~ N(0, I_rq)`` and ``A`` a seeded orthonormal ``d x rq`` basis per head.
  The historical stream shares ``A`` and uses its own draws.

Everything is drawn in float64 and then rounded once to the workload's element
type (bf16 or fp32). Arrays are token-major ``[B, N, H, d]``.
"""
from __future__ import annotations

import dataclasses

import numpy as np

N_MIX = 16
WITHIN_STD = 0.5
Q_DOMINANT_SCALE = 5.0

_S_PARAMS, _S_LABELS, _S_KNOISE, _S_VALUES = 0, 1, 2, 3
_S_Q_NOISE, _S_Q_U, _S_H_NOISE, _S_H_U = 4, 5, 6, 7


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    dtype: str            # "f32" or "bf16": element type of Q/K/V/O and tables
    batch: int
    heads: int
    head_dim: int
    n_cache: int          # packed cache length that the Query chunk attends over
    n_q: int              # Query chunk length
    q_start: int          # absolute position of the first Query token
    frame_tokens: int     # F: block-causal frame length inside the chunk
    n_centroids: int
    group_size: int
    rank: int
    top_m: int
    q_rank: int           # rank of the dominant Query subspace
    n_out: int            # outlier Key channels
    out_scale: float
    n_hist: int           # historical Queries for the second-moment statistics
    chunk: int            # tokens per append call
    seed: int
    kmeans_iters: int = 10
    storage: int = 0      # App. D.1 storage options: 1 = 8-bit group scales, 2 = retention gate, 4 = sparse rows
    metric: int = 0       # QSAC candidate metric: 0 = Eq. 9 (diagonal), 1 = the full quadratic form
    coef_rows: int = 0    # storage bit 2 (sparse PSAC rows): pool rows per head, 0 = one per slot
    coef_stage: int = 0   # storage bit 2: staging rows per head (largest append chunk), 0 = the chunk size
    q_align: float = 0.0  # > 0: the dominant Query directions load the Key outlier channels (weight in [0, 1])

    @property
    def capacity(self) -> int:
        return self.n_cache

    def chunks(self):
        """(start, length) of the append calls that fill the cache."""
        out, t = [], 0
        while t < self.n_cache:
            n = min(self.chunk, self.n_cache - t)
            out.append((t, n))
            t += n
        return out


def _w(name, **kw):
    return Workload(name=name, **kw)


WORKLOADS = {
    "tiny-f32": _w("tiny-f32", dtype="f32", batch=1, heads=2, head_dim=64,
                   n_cache=1024, n_q=256, q_start=768, frame_tokens=1,
                   n_centroids=16, group_size=32, rank=4, top_m=4, q_rank=4,
                   n_out=4, out_scale=10.0, n_hist=512, chunk=256, seed=0),
    "mg2-12h": _w("mg2-12h", dtype="bf16", batch=1, heads=12, head_dim=128,
                  n_cache=13200, n_q=2640, q_start=10560, frame_tokens=880,
                  n_centroids=64, group_size=32, rank=8, top_m=4, q_rank=8,
                  n_out=4, out_scale=10.0, n_hist=2640, chunk=2640, seed=1),
    "lingbot-40h": _w("lingbot-40h", dtype="bf16", batch=1, heads=40, head_dim=128,
                      n_cache=32760, n_q=4680, q_start=28080, frame_tokens=1560,
                      n_centroids=128, group_size=32, rank=16, top_m=4, q_rank=16,
                      n_out=4, out_scale=10.0, n_hist=4680, chunk=4680, seed=2),
    "batched-4x30h": _w("batched-4x30h", dtype="bf16", batch=4, heads=30, head_dim=128,
                        n_cache=24960, n_q=3120, q_start=21840, frame_tokens=1040,
                        n_centroids=256, group_size=64, rank=32, top_m=4, q_rank=32,
                        n_out=8, out_scale=20.0, n_hist=3120, chunk=3120, seed=4),
}
for _n in (30000, 60000, 120000):
    WORKLOADS[f"rollout-{_n // 1000}k"] = _w(
        f"rollout-{_n // 1000}k", dtype="bf16", batch=1, heads=40, head_dim=128,
        n_cache=_n, n_q=1560, q_start=_n - 1560, frame_tokens=1560,
        n_centroids=128, group_size=32, rank=16, top_m=4, q_rank=16,
        n_out=4, out_scale=10.0, n_hist=4680, chunk=4680, seed=3)


def scaled(wl: Workload, **changes) -> Workload:
    return dataclasses.replace(wl, **changes)


def _gen(wl: Workload, b: int, h: int, stream: int) -> np.random.Generator:
    key = np.array([(wl.seed << 24) ^ (b << 12) ^ h, stream], dtype=np.uint64)
    return np.random.Generator(np.random.Philox(key=key))


def _head_params(wl: Workload, b: int, h: int):
    g = _gen(wl, b, h, _S_PARAMS)
    d = wl.head_dim
    sigma = np.exp(g.standard_normal(d))
    out_ch = g.permutation(d)[: wl.n_out]
    sigma[out_ch] *= wl.out_scale
    means = sigma[None, :] * g.standard_normal((N_MIX, d))
    raw = g.standard_normal((d, wl.q_rank))
    if wl.q_align > 0:
        # the first dominant directions lean on the outlier channels of the Keys
        for i in range(min(wl.n_out, wl.q_rank)):
            unit = np.zeros(d)
            unit[out_ch[i]] = np.sqrt(d)
            raw[:, i] = wl.q_align * unit + (1.0 - wl.q_align) * raw[:, i]
    a, _ = np.linalg.qr(raw)
    return sigma, means, a


def keys_head(wl: Workload, b: int, h: int, n: int) -> np.ndarray:
    """float64 [n, d]: the first n Key tokens of head (b, h)."""
    sigma, means, _ = _head_params(wl, b, h)
    labels = _gen(wl, b, h, _S_LABELS).integers(0, N_MIX, size=n)
    noise = _gen(wl, b, h, _S_KNOISE).standard_normal((n, wl.head_dim))
    return means[labels] + WITHIN_STD * sigma[None, :] * noise


def values_head(wl: Workload, b: int, h: int, n: int) -> np.ndarray:
    return _gen(wl, b, h, _S_VALUES).standard_normal((n, wl.head_dim))


def queries_head(wl: Workload, b: int, h: int, n: int, historical: bool = False) -> np.ndarray:
    _, _, a = _head_params(wl, b, h)
    s_noise, s_u = (_S_H_NOISE, _S_H_U) if historical else (_S_Q_NOISE, _S_Q_U)
    noise = _gen(wl, b, h, s_noise).standard_normal((n, wl.head_dim))
    u = _gen(wl, b, h, s_u).standard_normal((n, wl.q_rank))
    return noise + Q_DOMINANT_SCALE * (u @ a.T)


def round_to(x: np.ndarray, dtype: str) -> np.ndarray:
    """Round float64 values to the element type; returns float32 holding them."""
    x32 = np.asarray(x, dtype=np.float32)
    if dtype == "f32":
        return x32
    if dtype != "bf16":
        raise ValueError(dtype)
    bits = x32.view(np.uint32).astype(np.uint64)
    lsb = (bits >> 16) & 1
    rounded = ((bits + 0x7FFF + lsb) >> 16) << 16
    return rounded.astype(np.uint32).view(np.float32)


def tensor(wl: Workload, what: str, n: int, start: int = 0, heads=None) -> np.ndarray:
    """float32 [B, n, H, d] of tokens [start, start + n) of one stream.

    ``what`` is "k", "v", "q" (the Query chunk) or "qhist". ``heads`` limits the
    work to a list of (b, h); other heads are left zero.
    """
    fn = {"k": keys_head, "v": values_head,
          "q": lambda w, b, h, m: queries_head(w, b, h, m, False),
          "qhist": lambda w, b, h, m: queries_head(w, b, h, m, True)}[what]
    out = np.zeros((wl.batch, n, wl.heads, wl.head_dim), dtype=np.float32)
    todo = heads if heads is not None else [(b, h) for b in range(wl.batch) for h in range(wl.heads)]
    for b, h in todo:
        out[b, :, h, :] = round_to(fn(wl, b, h, start + n)[start:], wl.dtype)
    return out
