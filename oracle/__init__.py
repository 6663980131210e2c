"""CPU oracle for the QuantWM hot path: TEST INFRASTRUCTURE ONLY.

Thin ctypes wrappers over ``libquantwm_oracle.so`` (plain C in
``quantwm_oracle.c``). Only ``tests/``, the package's ``smoke()`` check and the
benchmark's CPU-baseline leg may import this module; the product path never
does. Arrays are numpy float32 ``[B, N, H, d]`` holding values exact in the
workload's element type; method-level tables are float32 too.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(_HERE, "quantwm_oracle.c")
CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fopenmp", "-fPIC", "-shared",
          "-std=c11", "-Wall", "-Wextra"]
# QWM_ORACLE_SANITIZE=1: a build with AddressSanitizer and UndefinedBehaviorSanitizer
# (its own library file; the process must preload gcc's libasan, see
# tests/test_oracle_sanitized.py), any report fatal
SANITIZE = os.environ.get("QWM_ORACLE_SANITIZE") == "1"
if SANITIZE:
    CFLAGS = CFLAGS + ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]
LIB = os.path.join(_HERE, "libquantwm_oracle_san.so" if SANITIZE else "libquantwm_oracle.so")


def build() -> str:
    tmp = LIB + ".tmp"
    subprocess.run(["gcc", *CFLAGS, "-o", tmp, SRC, "-lm"], check=True)
    os.replace(tmp, LIB)
    return LIB


class OraCfg(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int), ("heads", ctypes.c_int), ("head_dim", ctypes.c_int),
                ("n_centroids", ctypes.c_int), ("group_size", ctypes.c_int),
                ("rank", ctypes.c_int), ("top_m", ctypes.c_int),
                ("capacity", ctypes.c_longlong), ("table_bf16", ctypes.c_int), ("storage", ctypes.c_int),
                ("metric", ctypes.c_int), ("coef_rows", ctypes.c_longlong), ("coef_stage", ctypes.c_longlong)]


# App. D.1 storage options (ORA_STORE_* in quantwm_oracle.h)
STORE_SCALE_I8 = 1
STORE_GATE = 2
STORE_SPARSE = 4
# QSAC candidate metric (ORA_METRIC_*): Eq. 9 or the full quadratic form
METRIC_DIAG = 0
METRIC_FULL = 1


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise RuntimeError(f"oracle library missing: {LIB} (run __graft_entry__.build())")
        _lib = ctypes.CDLL(LIB)
        _lib.ora_cache_bytes.restype = ctypes.c_longlong
        _lib.ora_coef_record_bytes.restype = ctypes.c_longlong
        _lib.ora_round_bf16.restype = ctypes.c_double
        _lib.ora_round_bf16.argtypes = [ctypes.c_double]
        _lib.ora_round_f16.restype = ctypes.c_double
        _lib.ora_round_f16.argtypes = [ctypes.c_double]
        _lib.ora_f16_bits.restype = ctypes.c_uint16
        _lib.ora_f16_bits.argtypes = [ctypes.c_double]
        _lib.ora_f16_value.restype = ctypes.c_double
        _lib.ora_f16_value.argtypes = [ctypes.c_uint16]
    return _lib


def cfg_of(batch, heads, head_dim, n_centroids, group_size, rank, top_m, capacity, bf16, storage=0,
           metric=0, coef_rows=0, coef_stage=0) -> OraCfg:
    return OraCfg(batch, heads, head_dim, n_centroids, group_size, rank, top_m, capacity, int(bf16), int(storage),
                  int(metric), int(coef_rows), int(coef_stage))


def cfg_from_workload(wl, capacity=None) -> OraCfg:
    return cfg_of(wl.batch, wl.heads, wl.head_dim, wl.n_centroids, wl.group_size, wl.rank,
                  wl.top_m, wl.capacity if capacity is None else capacity, wl.dtype == "bf16",
                  getattr(wl, "storage", 0), getattr(wl, "metric", 0), getattr(wl, "coef_rows", 0),
                  getattr(wl, "coef_stage", 0) or getattr(wl, "chunk", 0))


def _p(a, ct=ctypes.c_float):
    if a is None:
        return None
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ct))


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"oracle {what} failed with status {rc}")


def set_threads(n: int):
    lib().ora_set_threads(int(n))


def max_threads() -> int:
    return int(lib().ora_max_threads())


def cache_bytes(cfg: OraCfg) -> int:
    return int(lib().ora_cache_bytes(ctypes.byref(cfg)))


def token_bytes(cfg: OraCfg):
    kb, vb = ctypes.c_int(), ctypes.c_int()
    _check(lib().ora_token_bytes(ctypes.byref(cfg), ctypes.byref(kb), ctypes.byref(vb)), "token_bytes")
    return kb.value, vb.value


def round_bf16(x: float) -> float:
    return lib().ora_round_bf16(float(x))


def round_f16(x: float) -> float:
    return lib().ora_round_f16(float(x))


def f16_bits(x: float) -> int:
    return int(lib().ora_f16_bits(float(x)))


def f16_value(bits: int) -> float:
    return lib().ora_f16_value(int(bits))


def scales_i8(t):
    """App. D.1 8-bit group scales of one token-head: (sigma FP16 bits, codes, steps)."""
    t = _f32(t)
    ng = t.shape[0]
    codes = np.zeros(ng, np.uint8)
    steps = np.zeros(ng, np.float32)
    sig = ctypes.c_uint16(0)
    lib().ora_scales_i8(_p(t), ng, ctypes.byref(sig), _p(codes, ctypes.c_uint8), _p(steps))
    return int(sig.value), codes, steps


def int2_quantise(x, mu, step):
    """Eq. 1-2 and Eq. 4 of one group with a given (stored) step size."""
    x, mu = _f32(x), _f32(mu)
    n = x.shape[0]
    codes = np.zeros(n, np.uint8)
    xhat = np.zeros(n, np.float32)
    zp = ctypes.c_uint8(0)
    lib().ora_int2_quantise(_p(x), _p(mu), n, ctypes.c_float(step), _p(codes, ctypes.c_uint8),
                            ctypes.byref(zp), _p(xhat))
    return codes, int(zp.value), xhat


def coef_row(C):
    """App. D.1 INT8 PSAC row: (codes int8 [r], FP16 scale bits)."""
    C = _f32(C)
    codes = np.zeros(C.shape[0], np.int8)
    sb = ctypes.c_uint16(0)
    lib().ora_coef_row(_p(C), C.shape[0], _p(codes, ctypes.c_int8), ctypes.byref(sb))
    return codes, int(sb.value)


def keep_row(C, codes, scale, lam):
    """App. D.1 retention gate for one INT8 coefficient row."""
    C, lam = _f32(C), _f32(lam)
    codes = np.ascontiguousarray(codes, dtype=np.int8)
    return bool(lib().ora_keep_row(_p(C), _p(codes, ctypes.c_int8), ctypes.c_float(scale), _p(lam), C.shape[0]))


def int2_group(x, mu):
    x, mu = _f32(x), _f32(mu)
    n = x.shape[0]
    codes = np.zeros(n, np.uint8)
    zp, sc = ctypes.c_uint8(), ctypes.c_uint16()
    xhat = np.zeros(n, np.float32)
    lib().ora_int2_group(_p(x), _p(mu), n, _p(codes, ctypes.c_uint8), ctypes.byref(zp),
                         ctypes.byref(sc), _p(xhat))
    return codes, int(zp.value), int(sc.value), xhat


def qsac_assign(k, mu, w, group_size, top_m):
    k, mu, w = _f32(k), _f32(mu), _f32(w)
    kc, d = mu.shape
    cand = np.zeros(max(kc, 1), np.int32)
    z = lib().ora_qsac_assign(_p(k), _p(mu), _p(w), kc, d, group_size, top_m, _p(cand, ctypes.c_int))
    return int(z), cand[: min(top_m, kc)].copy()


def qsac_assign_full(k, mu, m, w, group_size, top_m):
    """QSAC with the candidates ranked by (k - mu)^T m (k - mu); m is [d, d]."""
    k, mu, m, w = _f32(k), _f32(mu), _f32(m), _f32(w)
    kc, d = mu.shape
    assert m.shape == (d, d)
    cand = np.zeros(max(kc, 1), np.int32)
    z = lib().ora_qsac_assign_full(_p(k), _p(mu), _p(m), _p(w), kc, d, group_size, top_m,
                                   _p(cand, ctypes.c_int))
    return int(z), cand[: min(top_m, kc)].copy()


def nearest(x, mu):
    x, mu = _f32(x), _f32(mu)
    return int(lib().ora_nearest(_p(x), _p(mu), mu.shape[0], mu.shape[1]))


def eigh(a):
    a = np.ascontiguousarray(a, dtype=np.float64)
    n = a.shape[0]
    lam = np.zeros(n)
    vt = np.zeros((n, n))
    _check(lib().ora_eigh(_p(a, ctypes.c_double), n, _p(lam, ctypes.c_double),
                          _p(vt, ctypes.c_double)), "eigh")
    return lam, vt


def calibrate(cfg: OraCfg, q_hist, k_cal, v_cal, kmeans_iters):
    """Returns (mu_k, mu_v, w, u_t, lam) as float32 arrays, and with the full
    metric (cfg.metric == METRIC_FULL) a sixth table: m [B, H, d, d], the Query
    second moment over the mean of its diagonal."""
    B, H, d, K, r = cfg.batch, cfg.heads, cfg.head_dim, cfg.n_centroids, cfg.rank
    q_hist = _f32(q_hist) if q_hist is not None else np.zeros((B, 0, H, d), np.float32)
    k_cal, v_cal = _f32(k_cal), _f32(v_cal)
    mu_k = np.zeros((B, H, K, d), np.float32)
    mu_v = np.zeros((B, H, K, d), np.float32)
    w = np.zeros((B, H, d), np.float32)
    u_t = np.zeros((B, H, max(r, 0), d), np.float32)
    lam = np.zeros((B, H, max(r, 0)), np.float32)
    full = cfg.metric == METRIC_FULL
    m = np.zeros((B, H, d, d), np.float32) if full else None
    rc = lib().ora_calibrate(ctypes.byref(cfg), _p(q_hist), ctypes.c_longlong(q_hist.shape[1]),
                             _p(k_cal), _p(v_cal), ctypes.c_longlong(k_cal.shape[1]), kmeans_iters,
                             _p(mu_k), _p(mu_v), _p(w), _p(u_t), _p(lam), _p(m))
    _check(rc, "calibrate")
    return (mu_k, mu_v, w, u_t, lam, m) if full else (mu_k, mu_v, w, u_t, lam)


def new_cache(cfg: OraCfg) -> np.ndarray:
    return np.zeros(cache_bytes(cfg), np.uint8)


def append(cfg: OraCfg, tables, cache, n_cached, k_new, v_new, diagnostics=False):
    """Writes slots [n_cached, n_cached + n) in place; returns diagnostics if asked.
    tables: (mu_k, mu_v, w, u_t[, lam[, m]]); m is read with the full metric only."""
    mu_k, mu_v, w, u_t = (_f32(t) for t in tables[:4])
    lam = _f32(tables[4]) if len(tables) > 4 and tables[4] is not None else None
    m = _f32(tables[5]) if len(tables) > 5 and tables[5] is not None else None
    k_new, v_new = _f32(k_new), _f32(v_new)
    B, n, H = k_new.shape[0], k_new.shape[1], k_new.shape[2]
    M = min(cfg.top_m, cfg.n_centroids)
    coef = np.zeros((B, H, n, max(cfg.rank, 1)), np.float32) if diagnostics else None
    kid = np.zeros((B, H, n), np.int32) if diagnostics else None
    vid = np.zeros((B, H, n), np.int32) if diagnostics else None
    cand = np.zeros((B, H, n, M), np.int32) if diagnostics else None
    rc = lib().ora_append(ctypes.byref(cfg), _p(mu_k), _p(mu_v), _p(w), _p(u_t), _p(lam), _p(m),
                          _p(cache, ctypes.c_uint8), ctypes.c_longlong(n_cached),
                          _p(k_new), _p(v_new), ctypes.c_longlong(n), _p(coef),
                          _p(kid, ctypes.c_int), _p(vid, ctypes.c_int), _p(cand, ctypes.c_int))
    _check(rc, "append")
    if diagnostics:
        return {"coef": coef[..., : cfg.rank], "k_ids": kid, "v_ids": vid, "cand": cand}
    return None


COEF_DENSE = 0
COEF_SPARSE = 1


def coef_record_bytes(cfg: OraCfg, cache, start, n):
    """(bytes, layout) of the chunk's coefficient record (App. D.1 layout choice)."""
    lay = ctypes.c_int()
    b = lib().ora_coef_record_bytes(ctypes.byref(cfg), _p(cache, ctypes.c_uint8), ctypes.c_longlong(start),
                                    ctypes.c_longlong(n), ctypes.byref(lay))
    if b < 0:
        raise RuntimeError("oracle coef_record_bytes failed")
    return int(b), int(lay.value)


def coef_pack(cfg: OraCfg, cache, start, n) -> np.ndarray:
    size, _ = coef_record_bytes(cfg, cache, start, n)
    out = np.zeros(size, np.uint8)
    wr = ctypes.c_longlong()
    _check(lib().ora_coef_pack(ctypes.byref(cfg), _p(cache, ctypes.c_uint8), ctypes.c_longlong(start),
                               ctypes.c_longlong(n), _p(out, ctypes.c_uint8), ctypes.c_longlong(size),
                               ctypes.byref(wr)), "coef_pack")
    assert wr.value == size
    return out


def coef_unpack(cfg: OraCfg, rec, cache, start, n):
    """Writes the record's rows into slots [start, start + n) of the cache in place."""
    rec = np.ascontiguousarray(rec, dtype=np.uint8)
    _check(lib().ora_coef_unpack(ctypes.byref(cfg), _p(rec, ctypes.c_uint8), ctypes.c_longlong(rec.size),
                                 _p(cache, ctypes.c_uint8), ctypes.c_longlong(start), ctypes.c_longlong(n)),
           "coef_unpack")


def decode(cfg: OraCfg, tables, cache, b, h, n):
    mu_k, mu_v = _f32(tables[0]), _f32(tables[1])
    d, r = cfg.head_dim, cfg.rank
    k0 = np.zeros((n, d)); v = np.zeros((n, d)); ch = np.zeros((n, max(r, 1)))
    rc = lib().ora_decode(ctypes.byref(cfg), _p(mu_k), _p(mu_v), _p(cache, ctypes.c_uint8), b, h,
                          ctypes.c_longlong(n), _p(k0, ctypes.c_double), _p(ch, ctypes.c_double),
                          _p(v, ctypes.c_double))
    _check(rc, "decode")
    return k0, ch[:, :r], v


def attend(cfg: OraCfg, tables, cache, n_cache, q, q_start, frame_tokens, rows=None,
           coef_override=None, want_logits=False, k_act=None, v_act=None, epochs=None):
    """rows: int array [n_rows, 3] of (b, h, i); default all rows. k_act / v_act
    ([B, n_act, H, d]) append an exact active chunk after the packed keys.
    epochs: optional list of (first key, tables) in increasing order, the first
    at key 0; packed keys then decode with their epoch's tables (`tables` unused).

    Returns (out [n_rows, d] fp64, lse [n_rows], logits [n_rows, n_cache + n_act] or None).
    """
    if epochs is None:
        epochs = [(0, tables)]
    starts = np.array([e[0] for e in epochs], np.int64)
    mu_k = np.ascontiguousarray(np.stack([_f32(e[1][0]) for e in epochs]))
    mu_v = np.ascontiguousarray(np.stack([_f32(e[1][1]) for e in epochs]))
    u_t = (np.ascontiguousarray(np.stack([_f32(e[1][3]) for e in epochs]))
           if cfg.rank > 0 and epochs[0][1][3] is not None else None)
    q = _f32(q)
    B, n_q, H, d = q.shape
    n_act = 0 if k_act is None else int(k_act.shape[1])
    ka = _f32(k_act) if k_act is not None else None
    va = _f32(v_act) if v_act is not None else None
    if rows is None:
        rows = np.array([(b, h, i) for b in range(B) for h in range(H) for i in range(n_q)], np.int32)
    rows = np.ascontiguousarray(rows, dtype=np.int32).reshape(-1, 3)
    nr = rows.shape[0]
    out = np.zeros((nr, d)); lse = np.zeros(nr)
    logits = np.zeros((nr, n_cache + n_act)) if want_logits else None
    co = _f32(coef_override) if coef_override is not None else None
    rc = lib().ora_attend_epochs(ctypes.byref(cfg), len(epochs), _p(starts, ctypes.c_longlong), _p(mu_k), _p(mu_v),
                                 _p(u_t), _p(cache, ctypes.c_uint8), ctypes.c_longlong(n_cache), _p(ka), _p(va),
                                 ctypes.c_longlong(n_act), _p(q), ctypes.c_longlong(n_q), ctypes.c_longlong(q_start),
                                 int(frame_tokens), _p(co), nr, _p(rows, ctypes.c_int), _p(out, ctypes.c_double),
                                 _p(lse, ctypes.c_double), _p(logits, ctypes.c_double))
    _check(rc, "attend")
    return out, lse, logits
