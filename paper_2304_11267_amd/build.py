"""Build libsdattn.so (the C ABI of include/sdattn.h) for gfx950 with hipcc.

Each csrc/*.hip file is compiled separately (in parallel) and linked into a
shared library in the package directory, where the binding loads it.  The
measurement kernels of include/sdattn_probes.h (csrc/probes.hip) go into a
library of their own, libsdattn_probes.so, which only the benchmark loads.
"""
from __future__ import annotations

import concurrent.futures
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libsdattn.so")
PROBES_LIB = os.path.join(HERE, "libsdattn_probes.so")
PROBE_SOURCES = ["probes.hip"]
ARCH = "gfx950"

SOURCES = ["attn_fwd.hip", "attn_fwd_bf16.hip", "attn_fwd_short.hip", "attn_fwd_generic.hip", "softmax_rows.hip",
           "twopass.hip", "linear.hip", "norm_act.hip", "winograd.hip",
           "sdattn_api.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Wall", "-Wno-unused-function",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
    # keep the compiler from emitting packed fp32 ops (v_pk_fma_f32 and friends)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # matrix-core results in ordinary VGPRs: the softmax reads them directly
    # instead of copying them out of accumulation registers
    "-mllvm", "-amdgpu-mfma-vgpr-form",
]

# Per-file additions.  The short-sequence kernel is latency-bound: its first 14
# argument dwords arrive preloaded in SGPRs instead of through scalar loads.
EXTRA_FLAGS = {
    "attn_fwd_short.hip": ["-mllvm", "-amdgpu-kernarg-preload-count=14"],
}


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *CFLAGS, *EXTRA_FLAGS.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError(f"hipcc failed on {src}")
    warn = "\n".join(l for l in r.stderr.splitlines() if "packed-fp32-ops" not in l
                     and "warning: feature flag" not in l and l.strip())
    if warn and verbose:
        sys.stderr.write(warn + "\n")
    return obj


def _link(objs, lib, verbose):
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = SOURCES + PROBE_SOURCES
    with concurrent.futures.ThreadPoolExecutor(max_workers=len(srcs)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), srcs))
    _link(objs[:len(SOURCES)], LIB, verbose)
    _link(objs[len(SOURCES):], PROBES_LIB, verbose)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
