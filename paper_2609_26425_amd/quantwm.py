"""ctypes binding of libquantwm.so: the QuantWM hot path on MI355X (gfx950).

Argument marshalling only: torch tensors become device pointers, the current
torch stream becomes the hipStream_t, and a non-zero status raises
QuantwmError. Every step of the path runs in the library's HIP kernels; there
is no fallback, and a missing library is an ImportError.
"""
from __future__ import annotations

import ctypes
import os

import torch

# QWM_LIB selects another build of the library (the sanitized host-side build
# that tests/test_abi_sanitized.py loads); by default the in-tree one
LIB_PATH = os.environ.get("QWM_LIB") or os.path.join(os.path.dirname(os.path.abspath(__file__)), "libquantwm.so")

F32, BF16 = 0, 1
OK, ERR_INVALID_ARG, ERR_UNSUPPORTED, ERR_CAPACITY, ERR_HIP = 0, 1, 2, 3, 4


class QuantwmError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"quantwm status {status}: {message}")
        self.status = status


class Config(ctypes.Structure):
    """Mirror of quantwm_config."""
    _fields_ = [("batch", ctypes.c_int32), ("heads", ctypes.c_int32), ("head_dim", ctypes.c_int32),
                ("n_centroids", ctypes.c_int32), ("group_size", ctypes.c_int32),
                ("rank", ctypes.c_int32), ("top_m", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("capacity", ctypes.c_int64), ("storage", ctypes.c_int32), ("metric", ctypes.c_int32),
                ("coef_rows", ctypes.c_int64), ("coef_stage", ctypes.c_int64)]

    @property
    def torch_dtype(self):
        return torch.bfloat16 if self.dtype == BF16 else torch.float32


class CalibLayout(ctypes.Structure):
    """Mirror of quantwm_calib_layout (byte offsets inside one (b, h) slab)."""
    _fields_ = [(n, ctypes.c_int64) for n in
                ("slab_bytes", "mu_k", "mu_v", "a_k", "b_k", "a_v", "b_v", "w", "wg", "u_t", "lam", "u_dr", "m",
                 "mu_k16", "mu_v16", "e16", "a_k3")]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with paper_2609_26425_amd/build.py "
                          "(or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    C = ctypes.POINTER(Config)
    sig = {
        "quantwm_cache_bytes": (SZ, [C]),
        "quantwm_token_bytes": (I32, [C, ctypes.POINTER(I32), ctypes.POINTER(I32)]),
        "quantwm_calib_bytes": (SZ, [C]),
        "quantwm_calib_offsets": (I32, [C, ctypes.POINTER(CalibLayout)]),
        "quantwm_calibrate_workspace_bytes": (SZ, [C, I64, I64]),
        "quantwm_calib_pack": (I32, [C, P, P, P, P, P, P, P, P]),
        "quantwm_calibrate": (I32, [C, P, I64, P, P, I64, I32, P, P, SZ, P]),
        "quantwm_stats_bytes": (SZ, [C]),
        "quantwm_stats_update": (I32, [C, P, I64, P, P]),
        "quantwm_calibrate_epoch": (I32, [C, P, P, P, I64, I32, P, P, SZ, P]),
        "quantwm_append": (I32, [C, P, P, I64, P, P, I64, P, P]),
        "quantwm_attend_workspace_bytes": (SZ, [C, I64, I64]),
        "quantwm_attend": (I32, [C, P, P, I64, P, I64, I64, I32, P, P, P, SZ, P]),
        "quantwm_attend_active": (I32, [C, P, P, I64, P, P, I64, P, I64, I64, I32, P, P, P, SZ, P]),
        "quantwm_attend_epochs": (I32, [C, P, I32, ctypes.POINTER(I64), P, I64, P, P, I64, P, I64, I64, I32, P, P,
                                        P, SZ, P]),
        "quantwm_logits": (I32, [C, P, P, I64, P, I64, I64, I64, I32, P, P]),
        "quantwm_attend_noalloc": (I32, [C, P, P, I64, P, I64, I64, I32, P, P, P]),
        "quantwm_attend_active_workspace_bytes": (SZ, [C, I64, I64, I64]),
        "quantwm_attend_epochs_workspace_bytes": (SZ, [C, I32, ctypes.POINTER(I64), I64, I64, I64]),
        "quantwm_coef_record_max_bytes": (SZ, [C, I64]),
        "quantwm_coef_pack": (I32, [C, P, I64, I64, P, SZ, ctypes.POINTER(I64), ctypes.POINTER(I32), P]),
        "quantwm_coef_unpack": (I32, [C, P, SZ, P, I64, I64, P]),
        "quantwm_coef_pool_usage": (I32, [C, P, I64, ctypes.POINTER(I64), ctypes.POINTER(I64), P]),
        "quantwm_last_error": (ctypes.c_char_p, []),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype, fn.argtypes = res, args
    return lib


_lib = _load()

EXPORTED = ("quantwm_cache_bytes", "quantwm_token_bytes", "quantwm_calib_bytes", "quantwm_calib_offsets",
            "quantwm_calibrate_workspace_bytes", "quantwm_calib_pack", "quantwm_calibrate", "quantwm_stats_bytes",
            "quantwm_stats_update", "quantwm_calibrate_epoch",
            "quantwm_append", "quantwm_attend_workspace_bytes", "quantwm_attend", "quantwm_attend_active",
            "quantwm_attend_epochs", "quantwm_attend_noalloc",
            "quantwm_logits", "quantwm_attend_active_workspace_bytes", "quantwm_attend_epochs_workspace_bytes", "quantwm_coef_record_max_bytes", "quantwm_coef_pack", "quantwm_coef_unpack",
            "quantwm_coef_pool_usage",
            "quantwm_last_error")


def library():
    return _lib


# App. D.1 storage options (QWM_STORE_* in include/quantwm.h)
STORE_SCALE_I8 = 1
STORE_GATE = 2
STORE_SPARSE = 4
# QSAC candidate metric (QWM_METRIC_*): Eq. 9 or the full quadratic form
METRIC_DIAG = 0
METRIC_FULL = 1


def make_config(batch, heads, head_dim, n_centroids, group_size, rank, top_m, capacity, dtype,
                storage=0, metric=0, coef_rows=0, coef_stage=0) -> Config:
    dt = {"bf16": BF16, "f32": F32, BF16: BF16, F32: F32}[dtype]
    return Config(batch, heads, head_dim, n_centroids, group_size, rank, top_m, dt, capacity, storage, metric,
                  coef_rows, coef_stage)


def _ptr(t):
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise TypeError("expected a torch.Tensor or None")
    if not t.is_contiguous():
        raise ValueError("tensors must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        if not torch.cuda.is_available():
            return None
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    if isinstance(stream, torch.cuda.Stream):
        return ctypes.c_void_p(stream.cuda_stream)
    return ctypes.c_void_p(int(stream))


def _check(status):
    if status != OK:
        raise QuantwmError(status, (_lib.quantwm_last_error() or b"").decode())


def quantwm_last_error() -> str:
    return (_lib.quantwm_last_error() or b"").decode()


def quantwm_cache_bytes(cfg: Config) -> int:
    return int(_lib.quantwm_cache_bytes(ctypes.byref(cfg)))


def quantwm_token_bytes(cfg: Config):
    k, v = ctypes.c_int32(), ctypes.c_int32()
    _check(_lib.quantwm_token_bytes(ctypes.byref(cfg), ctypes.byref(k), ctypes.byref(v)))
    return k.value, v.value


def quantwm_calib_bytes(cfg: Config) -> int:
    return int(_lib.quantwm_calib_bytes(ctypes.byref(cfg)))


def quantwm_calib_offsets(cfg: Config) -> CalibLayout:
    out = CalibLayout()
    _check(_lib.quantwm_calib_offsets(ctypes.byref(cfg), ctypes.byref(out)))
    return out


def quantwm_calibrate_workspace_bytes(cfg: Config, n_hist: int, n_calib: int) -> int:
    return int(_lib.quantwm_calibrate_workspace_bytes(ctypes.byref(cfg), n_hist, n_calib))


def quantwm_calib_pack(cfg, mu_k, mu_v, w, u_t, lam, calib, stream=None, m=None):
    """m: [B, H, d, d] float32, the matrix of the full metric (METRIC_FULL only)."""
    _check(_lib.quantwm_calib_pack(ctypes.byref(cfg), _ptr(mu_k), _ptr(mu_v), _ptr(w), _ptr(u_t), _ptr(lam),
                                   _ptr(m), _ptr(calib), _stream(stream)))


def quantwm_calibrate(cfg, q_hist, n_hist, k_calib, v_calib, n_calib, kmeans_iters, calib, workspace,
                      stream=None):
    _check(_lib.quantwm_calibrate(ctypes.byref(cfg), _ptr(q_hist), n_hist, _ptr(k_calib), _ptr(v_calib), n_calib,
                                  kmeans_iters, _ptr(calib), _ptr(workspace),
                                  0 if workspace is None else workspace.numel() * workspace.element_size(),
                                  _stream(stream)))


def quantwm_stats_bytes(cfg: Config) -> int:
    return int(_lib.quantwm_stats_bytes(ctypes.byref(cfg)))


def quantwm_stats_update(cfg, q, n, stats, stream=None):
    _check(_lib.quantwm_stats_update(ctypes.byref(cfg), _ptr(q), n, _ptr(stats), _stream(stream)))


def quantwm_calibrate_epoch(cfg, stats, k_calib, v_calib, n_calib, kmeans_iters, calib, workspace, stream=None):
    _check(_lib.quantwm_calibrate_epoch(ctypes.byref(cfg), _ptr(stats), _ptr(k_calib), _ptr(v_calib), n_calib,
                                        kmeans_iters, _ptr(calib), _ptr(workspace),
                                        0 if workspace is None else workspace.numel() * workspace.element_size(),
                                        _stream(stream)))


def quantwm_append(cfg, calib, cache, n_cached, k_new, v_new, n_new, coef_f32_out=None, stream=None):
    _check(_lib.quantwm_append(ctypes.byref(cfg), _ptr(calib), _ptr(cache), n_cached, _ptr(k_new), _ptr(v_new),
                               n_new, _ptr(coef_f32_out), _stream(stream)))


def quantwm_attend_workspace_bytes(cfg: Config, n_cache: int, n_q: int) -> int:
    return int(_lib.quantwm_attend_workspace_bytes(ctypes.byref(cfg), n_cache, n_q))


def quantwm_attend_active_workspace_bytes(cfg: Config, n_cache: int, n_act: int, n_q: int) -> int:
    return int(_lib.quantwm_attend_active_workspace_bytes(ctypes.byref(cfg), n_cache, n_act, n_q))


def quantwm_attend(cfg, calib, cache, n_cache, q, n_q, q_start, frame_tokens, out, lse_out=None, workspace=None,
                   stream=None):
    _check(_lib.quantwm_attend(ctypes.byref(cfg), _ptr(calib), _ptr(cache), n_cache, _ptr(q), n_q, q_start,
                               frame_tokens, _ptr(out), _ptr(lse_out), _ptr(workspace),
                               0 if workspace is None else workspace.numel() * workspace.element_size(),
                               _stream(stream)))


def quantwm_attend_active(cfg, calib, cache, n_cache, k_act, v_act, n_act, q, n_q, q_start, frame_tokens, out,
                          lse_out=None, workspace=None, stream=None):
    _check(_lib.quantwm_attend_active(ctypes.byref(cfg), _ptr(calib), _ptr(cache), n_cache, _ptr(k_act),
                                      _ptr(v_act), n_act, _ptr(q), n_q, q_start, frame_tokens, _ptr(out),
                                      _ptr(lse_out), _ptr(workspace),
                                      0 if workspace is None else workspace.numel() * workspace.element_size(),
                                      _stream(stream)))


def quantwm_attend_epochs(cfg, calibs, epoch_start, cache, n_cache, k_act, v_act, n_act, q, n_q, q_start,
                          frame_tokens, out, lse_out=None, workspace=None, stream=None):
    """calibs: one device buffer of len(epoch_start) calibration blocks; epoch_start: host ints."""
    starts = (ctypes.c_int64 * len(epoch_start))(*[int(x) for x in epoch_start])
    _check(_lib.quantwm_attend_epochs(ctypes.byref(cfg), _ptr(calibs), len(epoch_start), starts, _ptr(cache),
                                      n_cache, _ptr(k_act), _ptr(v_act), n_act, _ptr(q), n_q, q_start, frame_tokens,
                                      _ptr(out), _ptr(lse_out), _ptr(workspace),
                                      0 if workspace is None else workspace.numel() * workspace.element_size(),
                                      _stream(stream)))


def quantwm_attend_epochs_workspace_bytes(cfg, epoch_start, n_cache, n_act, n_q) -> int:
    starts = (ctypes.c_int64 * len(epoch_start))(*[int(x) for x in epoch_start])
    return int(_lib.quantwm_attend_epochs_workspace_bytes(ctypes.byref(cfg), len(epoch_start), starts, n_cache,
                                                          n_act, n_q))


ATTEND_NOALLOC_SCRATCH_BYTES = 128 << 20  # QWM_ATTEND_NOALLOC_SCRATCH_BYTES


def quantwm_attend_noalloc(cfg, calib, cache, n_cache, q, n_q, q_start, frame_tokens, out, lse_out=None,
                           stream=None):
    _check(_lib.quantwm_attend_noalloc(ctypes.byref(cfg), _ptr(calib), _ptr(cache), n_cache, _ptr(q), n_q, q_start,
                                       frame_tokens, _ptr(out), _ptr(lse_out), _stream(stream)))


def quantwm_logits(cfg, calib, cache, n_cache, q, n_q, q_start, frame_tokens, logits_out, stream=None, q_first=0):
    _check(_lib.quantwm_logits(ctypes.byref(cfg), _ptr(calib), _ptr(cache), n_cache, _ptr(q), n_q, q_start, q_first,
                               frame_tokens, _ptr(logits_out), _stream(stream)))


# App. D.1 per-chunk coefficient records (QWM_COEF_* in include/quantwm.h)
COEF_DENSE = 0
COEF_SPARSE = 1


def quantwm_coef_record_max_bytes(cfg, n) -> int:
    return int(_lib.quantwm_coef_record_max_bytes(ctypes.byref(cfg), n))


def quantwm_coef_pack(cfg, cache, start, n, record, stream=None):
    """Writes the chunk's coefficient record into the uint8 device tensor
    `record`; returns (bytes written, layout)."""
    written, layout = ctypes.c_int64(), ctypes.c_int32()
    _check(_lib.quantwm_coef_pack(ctypes.byref(cfg), _ptr(cache), start, n, _ptr(record), record.numel(),
                                  ctypes.byref(written), ctypes.byref(layout), _stream(stream)))
    return int(written.value), int(layout.value)


def quantwm_coef_unpack(cfg, record, cache, start, n, record_bytes=None, stream=None):
    nb = record.numel() if record_bytes is None else record_bytes
    _check(_lib.quantwm_coef_unpack(ctypes.byref(cfg), _ptr(record), nb, _ptr(cache), start, n, _stream(stream)))


def quantwm_coef_pool_usage(cfg, cache, n_cache, stream=None):
    """(rows used, rows dropped for lack of room) of a sparse-row cache."""
    used, dropped = ctypes.c_int64(), ctypes.c_int64()
    _check(_lib.quantwm_coef_pool_usage(ctypes.byref(cfg), _ptr(cache), n_cache, ctypes.byref(used),
                                        ctypes.byref(dropped), _stream(stream)))
    return int(used.value), int(dropped.value)
