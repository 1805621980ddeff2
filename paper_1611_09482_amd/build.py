"""Compile libfwg.so for gfx950 with hipcc (in-tree, next to this file)."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libfwg.so")
SOURCES = [os.path.join(CSRC, "fwg_host.cpp"), os.path.join(CSRC, "fwg_kernels.hip"),
           os.path.join(CSRC, "fwg_mfma.hip"), os.path.join(CSRC, "fwg_parallel.hip"),
           os.path.join(CSRC, "fwg_wave.hip"), os.path.join(CSRC, "fwg_split.hip"),
           os.path.join(CSRC, "fwg_chain.hip"), os.path.join(CSRC, "fwg_wide.hip")]
HEADERS = [os.path.join(ROOT, "include", "fwg.h"), os.path.join(CSRC, "fwg_internal.h"),
           os.path.join(CSRC, "fwg_sample.h"), os.path.join(CSRC, "fwg_valu.h"),
           os.path.join(CSRC, "fwg_wave.h"), os.path.join(CSRC, "fwg_par.h"), os.path.join(CSRC, "fwg_mfma_dev.h"),
           os.path.join(CSRC, "fwg_bf16.h"), os.path.join(CSRC, "fwg_chain.h"),
           os.path.join(CSRC, "fwg_xchg.h"), os.path.join(CSRC, "fwg_wide.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # packed fp32 instructions stay off: the compiler must not form them from float code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary VGPRs: avoids AGPR<->VGPR copies around the step loop
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
]
OBJDIR = os.path.join(PKG, "_build")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("hipcc failed: " + " ".join(cmd[-3:]))


def build(verbose: bool = False) -> str:
    """Compile every source to an object (in parallel: each is one translation unit with its own
    device code), then link libfwg.so."""
    os.makedirs(OBJDIR, exist_ok=True)
    objs = [os.path.join(OBJDIR, os.path.basename(src) + ".o") for src in SOURCES]
    jobs = max(1, min(len(SOURCES), int(os.environ.get("MAX_JOBS", os.cpu_count() or 1))))
    with ThreadPoolExecutor(jobs) as ex:
        for f in [ex.submit(_run, [HIPCC] + FLAGS + ["-c", "-o", o, src], verbose) for src, o in zip(SOURCES, objs)]:
            f.result()
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs, verbose)
    os.replace(tmp, LIB)
    return LIB


def is_stale() -> bool:
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(s) > t for s in SOURCES + HEADERS)


if __name__ == "__main__":
    print(build(verbose=True))
