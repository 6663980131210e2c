"""Builds libquantwm.so (the gfx950 HIP kernels plus the C ABI) in-tree.

Translation units compile in parallel: append.hip (fp32) and append_bf16.hip
once per (head_dim, group size), attend.hip once per (element type, head_dim, PSAC rank padding),
attend_host.hip, calib.hip, coef.hip, api.hip and the host eigensolver; the
objects link into ``paper_2609_26425_amd/libquantwm.so``.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libquantwm.so")
BUILD = os.path.join(HERE, "_build")
ARCH = os.environ.get("QWM_OFFLOAD_ARCH", "gfx950")

# -ffp-contract=off: every a*b+c that is not an explicit fma is two roundings, as
# the quantiser's integer decisions require. Packed FP32 arithmetic is disabled: the
# kernels are written for non-packed fp32 vector operations.
HIPFLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-ffp-contract=off",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops", "-Wall",
            "-Wno-unused-function"]


def _units():
    units = []
    # append_bf16: no NaN semantics either (its inputs are finite), so the group
    # ranges are v_min/v_max rather than compare-and-select pairs
    for tn, src, extra in (("f32", "append.hip", []), ("bf16", "append_bf16.hip", ["-fno-honor-nans"])):
        for d in (64, 128):
            for g in (16, 32, 64):
                units.append((f"append_{tn}_{d}_g{g}.o", src,
                              extra + [f"-DQWM_APPEND_D={d}", f"-DQWM_APPEND_G={g}"]))
    # attend: no NaN semantics, so maxima of matrix-core results are plain
    # v_max3_f32 without a quieting v_max_f32 x, x per input (its logits and
    # running maxima are finite or -inf). One unit per (element type, head_dim,
    # PSAC rank padding), so the instances compile in parallel.
    for tn, t in (("f32", "float"), ("bf16", "qwm::bf16")):
        for d in (64, 128):
            for rp in (0, 16, 32):
                units.append((f"attend_{tn}_{d}_r{rp}.o", "attend.hip",
                              ["-fno-honor-nans", f"-DQWM_ATTEND_T={t}", f"-DQWM_ATTEND_D={d}",
                               f"-DQWM_ATTEND_RP={rp}"]))
    units.append(("attend_host.o", "attend_host.hip", ["-fno-honor-nans"]))
    for name in ("calib", "coef", "api"):
        units.append((f"{name}.o", f"{name}.hip", []))
    units.append(("eigh.o", "eigh.cpp", ["-x", "hip"]))
    return units


def _hipcc():
    return shutil.which("hipcc") or "/opt/rocm/bin/hipcc"


def _compile(obj, src, extra):
    cmd = [_hipcc(), *HIPFLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", os.path.join(BUILD, obj)]
    p = subprocess.run(cmd, capture_output=True, text=True)
    errs = "\n".join(l for l in p.stderr.splitlines() if "is not a recognized feature" not in l)
    if p.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src} {extra}:\n{errs}")
    return obj


def _stale(obj, src):
    """True when the object is missing or older than its source or a header."""
    o = os.path.join(BUILD, obj)
    if not os.path.exists(o):
        return True
    deps = [os.path.join(CSRC, src)] + [os.path.join(CSRC, h) for h in os.listdir(CSRC) if h.endswith(".h")]
    deps.append(os.path.join(HERE, "..", "include", "quantwm.h"))
    return any(os.path.getmtime(p) > os.path.getmtime(o) for p in deps)


def build(jobs: int | None = None, verbose: bool = False, incremental: bool = False) -> str:
    """Compiles every unit (or, with incremental, only those older than their
    sources) and links the library."""
    os.makedirs(BUILD, exist_ok=True)
    units = _units()
    todo = [u for u in units if not incremental or _stale(u[0], u[1])]
    jobs = jobs or min(len(units), max(1, min(os.cpu_count() or 1, 16)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        futs = [ex.submit(_compile, *u) for u in todo]
        for f in cf.as_completed(futs):
            obj = f.result()
            if verbose:
                print("built", obj, flush=True)
    tmp = OUT + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp,
           *[os.path.join(BUILD, u[0]) for u in units]]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    os.replace(tmp, OUT)
    return OUT


SAN_OUT = os.path.join(BUILD, "san", "libquantwm_san.so")


def build_sanitized() -> str:
    """libquantwm with its host-side code (the C ABI's validation and launches,
    the host eigensolver) built with AddressSanitizer and UndefinedBehaviorSanitizer,
    linked with the kernel objects of the normal build (built first if missing).
    A process that loads it must preload clang's ASan runtime."""
    units = _units()
    if any(not os.path.exists(os.path.join(BUILD, u[0])) for u in units):
        build()
    san = os.path.join(BUILD, "san")
    os.makedirs(san, exist_ok=True)
    flags = ["-Xarch_host", "-fsanitize=address,undefined", "-Xarch_host", "-fno-sanitize-recover=all",
             "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
    objs = []
    for obj, src, extra in units:
        if src in ("api.hip", "eigh.cpp"):
            out = os.path.join(san, obj)
            cmd = [_hipcc(), *HIPFLAGS, *extra, *flags, "-c", os.path.join(CSRC, src), "-o", out]
            p = subprocess.run(cmd, capture_output=True, text=True)
            if p.returncode != 0:
                raise RuntimeError(f"hipcc failed for {src} (sanitized):\n{p.stderr}")
            objs.append(out)
        else:
            objs.append(os.path.join(BUILD, obj))
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-Xarch_host", "-fsanitize=address,undefined",
           "-shared-libsan", "-o", SAN_OUT, *objs]
    subprocess.run(cmd, check=True, capture_output=True, text=True)
    return SAN_OUT


if __name__ == "__main__":
    print(build(verbose=True, incremental="--incremental" in sys.argv))
    sys.exit(0)
