"""Build libisc.so (the HIP library behind include/isc.h) for gfx950.

    python -m paper_1704_07724_amd.build

Every .hip file under csrc/ is compiled by hipcc to an object in _build/ and
linked into paper_1704_07724_amd/libisc.so, next to the Python binding that
loads it.  Packed fp32 VALU instructions are disabled for all device code.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import re
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libisc.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

DEVICE_FLAGS = [
    "--offload-arch=" + ARCH,
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-result",
    # no packed fp32 VALU ops anywhere in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
]


# Per-file extra flags.  The register-tile kernels (sparse_reg, sparse_res,
# sparse_fused) keep accumulator tiles in registers through a compile-time
# dispatch tree on a wave-uniform value:
#  - SimplifyCFG's sinking of the common tails of the tree's leaves turns
#    constant register indices into selected pointers and forces the tile to
#    scratch memory, so sinking is disabled;
#  - every branch of the tree is uniform, so the CFG structurizer is told to
#    leave uniform regions alone (otherwise its flow blocks add scalar work
#    per level and break the in-place accumulate into copy chains).
_TILE_FLAGS = ["-mllvm", "-simplifycfg-sink-common=false",
               "-mllvm", "-structurizecfg-skip-uniform-regions"]
FILE_FLAGS = {"sparse_reg.hip": _TILE_FLAGS, "sparse_res.hip": _TILE_FLAGS, "sparse_fused.hip": _TILE_FLAGS}


def _spills(remarks: str) -> list:
    """Kernels whose resource-usage remark reports scratch (register spills
    or stack) -- a performance bug for the register-tile kernels."""
    out, name = [], None
    for line in remarks.splitlines():
        m = re.search(r"Function Name: (\S+)", line)
        if m:
            name = m.group(1)
        m = re.search(r"ScratchSize \[bytes/lane\]: (\d+)", line)
        if m and name and int(m.group(1)) > 0:
            out.append((name, int(m.group(1))))
    return out


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = ([HIPCC] + DEVICE_FLAGS + FILE_FLAGS.get(os.path.basename(src), []) +
           ["-Rpass-analysis=kernel-resource-usage", "-c", src, "-o", obj])
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr))
    for name, size in _spills(r.stderr):
        sys.stderr.write("warning: %s: kernel %s uses %d bytes of scratch per lane\n"
                         % (os.path.basename(src), name, size))
    warn = "\n".join(l for l in r.stderr.splitlines()
                     if "packed-fp32-ops" not in l and "kernel-resource-usage" not in l
                     and "remark:" not in l and l.strip())
    if warn:
        sys.stderr.write(warn + "\n")
    return obj


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link libisc.so; returns its path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    sources = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    if not sources:
        raise RuntimeError("no HIP sources under " + CSRC)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(sources))) as ex:
        objs = list(ex.map(_compile, sources))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr))
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
