"""Compile the HIP library (kernels + C ABI) for gfx950 with hipcc."""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "liblce.so")
# One translation unit per kernel family, compiled in parallel, then linked.
SOURCES = [os.path.join(CSRC, f) for f in ("lce.hip", "mfma_tiles.hip", "mfma_fs.hip",
                                                  "mfma_fs_win.hip", "quant_conv.hip")]
BUILD_DIR = os.path.join(PKG, "_build")
# Measurement-only probe of the xor/popcount VALU rate (not part of the C ABI).
PROBE_LIB = os.path.join(PKG, "libprobe.so")
PROBE_SOURCES = [os.path.join(CSRC, "valu_probe.hip")]
HEADERS = [os.path.join(CSRC, f) for f in ("bitpack.hpp", "bconv.hpp", "pool.hpp",
                                                 "bconv_mfma.hpp", "launch.hpp", "mfma_fs_launch.hpp", "dpp.hpp",
                                                 "bconv_quant.hpp")] + \
          [os.path.join(INCLUDE, "lce.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # Packed-fp32 VALU forms stay off (plain fp32 code only).
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def _compile(sources, lib, verbose, extra=()):
    """Compile each source to an object (in parallel), then link the shared
    library; the result replaces `lib` atomically."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    tag = f"{os.path.basename(lib)}.{os.getpid()}"
    objs = [os.path.join(BUILD_DIR, f"{os.path.basename(src)}.{tag}.o") for src in sources]
    cmds = [[HIPCC, *FLAGS, *extra, "-I", INCLUDE, "-I", CSRC, "-c", "-o", o, src]
            for src, o in zip(sources, objs)]
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(len(cmds), 8)) as ex:
        for f in [ex.submit(_run, c, verbose) for c in cmds]:
            f.result()
    tmp = lib + f".tmp{os.getpid()}"
    _run([HIPCC, *FLAGS, *extra, "-shared", "-o", tmp, *objs], verbose)
    os.replace(tmp, lib)
    for o in objs:
        os.remove(o)


def build(verbose: bool = False, extra=()) -> str:
    _compile(SOURCES, LIB, verbose, extra)
    _compile(PROBE_SOURCES, PROBE_LIB, verbose, extra)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB) or not os.path.exists(PROBE_LIB):
        return True
    t = min(os.path.getmtime(LIB), os.path.getmtime(PROBE_LIB))
    return any(os.path.getmtime(f) > t for f in SOURCES + HEADERS + PROBE_SOURCES)


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
