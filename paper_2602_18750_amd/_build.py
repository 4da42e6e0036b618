"""Build libhill.so (HIP, gfx950) in-tree with hipcc.

Usage: python -m paper_2602_18750_amd._build [-v]
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libhill.so")
# the benchmark's roofline calibration read, a library of its own (not libhill's ABI)
CALIB_LIB = os.path.join(PKG, "libhill_calib.so")
# the same library with its host layer (hill_api.cpp: validation, workspace
# layouts, launch set-up) built with AddressSanitizer and UBSan, for CPU runs
# of the error paths with the sanitizer runtime preloaded; device code as in LIB
HOSTSAN_LIB = os.path.join(PKG, "libhill_hostsan.so")
# host-only sanitizer flags (each behind -Xarch_host: no GPU code is instrumented)
HOSTSAN_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer"] + [
    x for f in ("-fsanitize=address", "-fsanitize=undefined", "-fno-sanitize-recover=all") for x in ("-Xarch_host", f)]
# per-kernel registers, scratch and occupancy as the compiler reports them
RESOURCES = os.path.join(BUILD_DIR, "kernel_resources.txt")

SOURCES = ["hill_api.cpp", "score.hip", "update.hip", "sketch.hip", "topk.hip", "attn.hip", "bkp.hip", "noalloc.hip", "tier.hip"]
CALIB_SOURCES = ["calib.hip"]
ARCH = os.environ.get("HILL_OFFLOAD_ARCH", "gfx950")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
COMMON = ["-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden", "--offload-arch=" + ARCH,
          # packed fp32 instructions stay disabled on gfx950
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-Wall", "-Wno-unused-result", "-I", INCLUDE, "-I", CSRC]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip", "-Rpass-analysis=kernel-resource-usage"] if src.endswith(".hip") else []
    cmd = [HIPCC] + COMMON + lang + ["-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    lines = (r.stderr or "").splitlines()
    usage = [l for l in lines if "kernel-resource-usage" in l]
    errs = "\n".join(l for l in lines if "packed-fp32-ops" not in l and "kernel-resource-usage" not in l)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed on %s:\n%s" % (src, errs))
    if verbose and errs.strip():
        print(errs, flush=True)
    with open(os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".resources"), "w") as f:
        f.write("\n".join(usage) + "\n")
    return obj


def _resource_report():
    """One line per kernel: name, VGPRs, scratch bytes per lane, occupancy."""
    rows = []
    for src in SOURCES + CALIB_SOURCES:
        path = os.path.join(BUILD_DIR, os.path.splitext(src)[0] + ".resources")
        if not src.endswith(".hip") or not os.path.exists(path):
            continue
        cur = {}
        for line in open(path):
            body = line.split("remark: ", 1)[-1].split(" [-Rpass", 1)[0].strip()
            key, _, val = body.partition(":")
            key, val = key.strip(), val.strip()
            if key == "Function Name":
                cur = {"name": val, "src": src}
                rows.append(cur)
            elif key in ("VGPRs", "ScratchSize [bytes/lane]", "Occupancy [waves/SIMD]"):
                cur[key.split()[0]] = val
    with open(RESOURCES, "w") as f:
        for r in rows:
            f.write("%s\t%s\tvgpr=%s\tscratch=%s\toccupancy=%s\n" % (
                r["src"], r["name"], r.get("VGPRs", "?"), r.get("ScratchSize", "?"), r.get("Occupancy", "?")))
    return rows


def _link(objs, lib, verbose):
    tmp = lib + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s" % r.stderr)
    os.replace(tmp, lib)


def build_host_sanitized(verbose: bool = False) -> str:
    """HOSTSAN_LIB from hill_api.cpp built with the sanitizers and the regular
    build's device objects (run build() first)."""
    objs = [os.path.join(BUILD_DIR, os.path.splitext(s)[0] + ".o") for s in SOURCES if s != "hill_api.cpp"]
    missing = [o for o in objs if not os.path.exists(o)]
    if missing:
        raise RuntimeError("build() first: missing %s" % ", ".join(missing))
    obj = os.path.join(BUILD_DIR, "hill_api_hostsan.o")
    cmd = [HIPCC] + COMMON + HOSTSAN_FLAGS + ["-c", os.path.join(CSRC, "hill_api.cpp"), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed on hill_api.cpp (sanitized):\n%s" % r.stderr)
    _link([obj] + objs, HOSTSAN_LIB, verbose)
    return HOSTSAN_LIB


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = SOURCES + CALIB_SOURCES
    with ThreadPoolExecutor(max_workers=len(srcs)) as ex:
        objs = dict(zip(srcs, ex.map(lambda s: _compile(s, verbose), srcs)))
    _link([objs[s] for s in SOURCES], LIB, verbose)
    _link([objs[s] for s in CALIB_SOURCES], CALIB_LIB, verbose)
    _resource_report()
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv[1:]))
