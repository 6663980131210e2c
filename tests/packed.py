"""Reads the packed cache format documented in include/quantwm.h into numpy
fields, for comparing caches byte-field by byte-field in tests."""
from __future__ import annotations

import numpy as np


def _up256(x):
    return (x + 255) // 256 * 256


def layout(batch, heads, d, G, r, capacity, storage=0, coef_rows=0, coef_stage=0):
    """storage bit 0: group scales as 8-bit codes plus an FP16 secondary scale
    per token (sections k_sigma / v_sigma at the end). Bit 2: sparse PSAC rows,
    K coef / K cscale hold a pool of coef_rows rows per head (all slots when 0),
    followed at the end by the tile directory and the overflow counters."""
    ng = d // G
    zpb = (ng + 3) // 4
    slots = (capacity + 63) // 64 * 64
    bh = batch * heads
    i8 = bool(storage & 1)
    sparse = bool(storage & 4)
    pool = coef_rows if sparse and coef_rows > 0 else slots
    sb = ng if i8 else 2 * ng
    per = [("k_codes", slots, d // 4), ("k_ids", slots, 1), ("k_zp", slots, zpb), ("k_scale", slots, sb),
           ("k_coef", pool, r), ("k_cscale", pool, 2 if r > 0 else 0), ("v_codes", slots, d // 4),
           ("v_ids", slots, 1), ("v_zp", slots, zpb), ("v_scale", slots, sb), ("k_sigma", slots, 2 if i8 else 0),
           ("v_sigma", slots, 2 if i8 else 0), ("k_dir", slots // 64, 16 if sparse else 0),
           ("k_over", 1, 4 if sparse else 0), ("k_st_codes", coef_stage if sparse else 0, r),
           ("k_st_scale", coef_stage if sparse else 0, 2)]
    off, nrows, at = {}, {}, 0
    for name, rows, nbytes in per:
        off[name] = (at, nbytes)
        nrows[name] = rows
        at = _up256(at + bh * rows * nbytes)
    return {"off": off, "rows": nrows, "slots": slots, "total": at, "ng": ng, "zpb": zpb, "d": d, "r": r,
            "bh": bh, "i8": i8, "sparse": sparse, "pool": pool}


def directory(buf: np.ndarray, lay, bh: int):
    """Sparse rows: (base [tiles] u32, mask [tiles] u64) of head bh's tile directory."""
    o, nb = lay["off"]["k_dir"]
    tiles = lay["slots"] // 64
    ent = np.asarray(buf, np.uint8)[o + bh * tiles * 16: o + (bh + 1) * tiles * 16].reshape(tiles, 16)
    base = np.ascontiguousarray(ent[:, 0:4]).view("<u4")[:, 0]
    mask = np.ascontiguousarray(ent[:, 8:16]).view("<u8")[:, 0]
    return base, mask


def pool(buf: np.ndarray, lay, bh: int):
    """Sparse rows: (codes [pool, r] int8, scale bits [pool] u16) of head bh's pool."""
    P, r = lay["pool"], lay["r"]
    oc, _ = lay["off"]["k_coef"]
    os_, _ = lay["off"]["k_cscale"]
    b = np.asarray(buf, np.uint8)
    codes = b[oc + bh * P * r: oc + (bh + 1) * P * r].reshape(P, r).view(np.int8)
    scale = np.ascontiguousarray(b[os_ + bh * P * 2: os_ + (bh + 1) * P * 2]).view("<u2")
    return codes, scale


def overflow(buf: np.ndarray, lay, bh: int) -> int:
    o, _ = lay["off"]["k_over"]
    return int(np.ascontiguousarray(np.asarray(buf, np.uint8)[o + 4 * bh: o + 4 * bh + 4]).view("<u4")[0])


def fields(buf: np.ndarray, lay, bh: int, t0: int, t1: int):
    """Fields of tokens [t0, t1) of flattened head bh."""
    buf = np.asarray(buf, dtype=np.uint8)
    s = lay["slots"]
    out = {}
    for name, (o, nb) in lay["off"].items():
        if nb == 0 or name in ("k_dir", "k_over", "k_st_codes", "k_st_scale") or \
                (lay.get("sparse") and name in ("k_coef", "k_cscale")):
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
    if r > 0 and not lay.get("sparse"):
        res["k_coef"] = np.ascontiguousarray(out["k_coef"]).view(np.int8)
        res["k_cscale"] = np.ascontiguousarray(out["k_cscale"]).view(np.uint16)[:, 0]
    elif r > 0:
        # a slot's row through the tile directory; a slot without one reads as zeros
        base, mask = directory(buf, lay, bh)
        codes, scale = pool(buf, lay, bh)
        kc = np.zeros((t1 - t0, r), np.int8)
        ks = np.zeros(t1 - t0, np.uint16)
        for j, t in enumerate(range(t0, t1)):
            T, i = divmod(t, 64)
            m = int(mask[T])
            if (m >> i) & 1:
                row = int(base[T]) + bin(m & ((1 << i) - 1)).count("1")
                kc[j], ks[j] = codes[row], scale[row]
        res["k_coef"], res["k_cscale"] = kc, ks
    return res


def copy_head(dst: np.ndarray, dst_lay, dst_bh: int, src: np.ndarray, src_lay, src_bh: int, n: int):
    """Byte copy of slots [0, n) of one head between two caches of the same format
    (with sparse rows: the head's whole pool, directory and overflow counter)."""
    for name, (o_d, nb) in dst_lay["off"].items():
        if nb == 0:
            continue
        o_s, _ = src_lay["off"][name]
        sd, ss = dst_lay["rows"][name], src_lay["rows"][name]
        cnt = n if sd == dst_lay["slots"] else min(sd, ss)
        dst[o_d + dst_bh * sd * nb: o_d + (dst_bh * sd + cnt) * nb] = \
            src[o_s + src_bh * ss * nb: o_s + (src_bh * ss + cnt) * nb]


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
