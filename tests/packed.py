"""Reads the packed cache format documented in include/quantwm.h into numpy
fields, for comparing caches byte-field by byte-field in tests."""
from __future__ import annotations

import numpy as np


def _up256(x):
    return (x + 255) // 256 * 256


def layout(batch, heads, d, G, r, capacity, storage=0):
    """storage bit 0: group scales as 8-bit codes plus an FP16 secondary scale
    per token (sections k_sigma / v_sigma at the end)."""
    ng = d // G
    zpb = (ng + 3) // 4
    slots = (capacity + 63) // 64 * 64
    rows = batch * heads * slots
    i8 = bool(storage & 1)
    sb = ng if i8 else 2 * ng
    per = [("k_codes", d // 4), ("k_ids", 1), ("k_zp", zpb), ("k_scale", sb), ("k_coef", r),
           ("k_cscale", 2 if r > 0 else 0), ("v_codes", d // 4), ("v_ids", 1), ("v_zp", zpb),
           ("v_scale", sb), ("k_sigma", 2 if i8 else 0), ("v_sigma", 2 if i8 else 0)]
    off, at = {}, 0
    for name, nbytes in per:
        off[name] = (at, nbytes)
        at = _up256(at + rows * nbytes)
    return {"off": off, "slots": slots, "total": at, "ng": ng, "zpb": zpb, "d": d, "r": r,
            "bh": batch * heads, "i8": i8}


def fields(buf: np.ndarray, lay, bh: int, t0: int, t1: int):
    """Fields of tokens [t0, t1) of flattened head bh."""
    buf = np.asarray(buf, dtype=np.uint8)
    s = lay["slots"]
    out = {}
    for name, (o, nb) in lay["off"].items():
        if nb == 0:
            continue
        seg = buf[o + (bh * s + t0) * nb: o + (bh * s + t1) * nb].reshape(t1 - t0, nb)
        out[name] = seg
    d, ng, r = lay["d"], lay["ng"], lay["r"]
    res = {}
    for p in ("k", "v"):
        codes = out[f"{p}_codes"]
        res[f"{p}_codes"] = np.stack([(codes >> (2 * i)) & 3 for i in range(4)], -1).reshape(t1 - t0, d)
        res[f"{p}_ids"] = out[f"{p}_ids"][:, 0].astype(np.int32)
        zp = out[f"{p}_zp"].astype(np.uint32)
        zw = sum(zp[:, i] << (8 * i) for i in range(zp.shape[1]))
        res[f"{p}_zp"] = np.stack([(zw >> (2 * g)) & 3 for g in range(ng)], -1)
        if lay.get("i8"):
            res[f"{p}_scale"] = np.ascontiguousarray(out[f"{p}_scale"]).reshape(t1 - t0, ng)
            res[f"{p}_sigma"] = np.ascontiguousarray(out[f"{p}_sigma"]).view(np.uint16)[:, 0]
        else:
            res[f"{p}_scale"] = np.ascontiguousarray(out[f"{p}_scale"]).view(np.uint16).reshape(t1 - t0, ng)
    if r > 0:
        res["k_coef"] = np.ascontiguousarray(out["k_coef"]).view(np.int8)
        res["k_cscale"] = np.ascontiguousarray(out["k_cscale"]).view(np.uint16)[:, 0]
    return res


def copy_head(dst: np.ndarray, dst_lay, dst_bh: int, src: np.ndarray, src_lay, src_bh: int, n: int):
    """Byte copy of slots [0, n) of one head between two caches of the same format."""
    for name, (o_d, nb) in dst_lay["off"].items():
        if nb == 0:
            continue
        o_s, _ = src_lay["off"][name]
        sd, ss = dst_lay["slots"], src_lay["slots"]
        dst[o_d + dst_bh * sd * nb: o_d + (dst_bh * sd + n) * nb] = \
            src[o_s + src_bh * ss * nb: o_s + (src_bh * ss + n) * nb]


def zero_coef_rows(buf: np.ndarray, lay, bh: int, slots):
    """Zero the PSAC codes and scale of the given slots of head bh (a dropped row)."""
    s = lay["slots"]
    (oc, nc), (os_, ns) = lay["off"]["k_coef"], lay["off"]["k_cscale"]
    for t in slots:
        buf[oc + (bh * s + t) * nc: oc + (bh * s + t + 1) * nc] = 0
        buf[os_ + (bh * s + t) * ns: os_ + (bh * s + t + 1) * ns] = 0


def coef_byte_mask(lay, nbh: int, start: int, n: int) -> np.ndarray:
    """Mask of the cache bytes holding the PSAC codes and scales of slots
    [start, start + n) of every head."""
    m = np.zeros(lay["total"], bool)
    s = lay["slots"]
    for name in ("k_coef", "k_cscale"):
        o, nb = lay["off"][name]
        for bh in range(nbh):
            m[o + (bh * s + start) * nb: o + (bh * s + start + n) * nb] = True
    return m
