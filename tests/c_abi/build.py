"""Build step for the plain-C client of the C ABI (test infrastructure).

Compiles ``closed_forms.c`` with gcc against ``include/sdattn.h`` and the HIP
runtime, linked to the in-tree ``libsdattn.so`` (found at run time through an
rpath relative to the executable).  Needs the library built first.
"""
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
SRC = os.path.join(HERE, "closed_forms.c")
EXE = os.path.join(HERE, "closed_forms")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build(verbose: bool = False) -> str:
    tmp = EXE + ".tmp"
    cmd = ["gcc", "-std=c11", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           SRC, "-o", tmp,
           "-L", os.path.join(ROOT, "paper_2304_11267_amd"), "-lsdattn",
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-lm",
           "-Wl,-rpath,$ORIGIN/../../paper_2304_11267_amd", "-Wl,-rpath," + os.path.join(ROCM, "lib")]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, EXE)
    return EXE


if __name__ == "__main__":
    print(build(verbose=True))
