"""Build the HIP library (libnf.so) for gfx950 in-tree with hipcc.

    python -m paper_1902_06714_amd.build

Always recompiles; the library lands next to this file.

One process must hold one HIP runtime.  PyTorch's ROCm wheel carries its own
copy of the runtime (soname libamdhip64.so.7, the same as ROCm's), which its
libraries request by the unversioned file name.  A process that loads torch
first therefore satisfies this library's libamdhip64.so.7 with torch's copy;
loading this library first would pull in ROCm's copy and torch would then add
a second one.  The Python binding imports torch before loading the library.
"""

from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libnf.so")
SOURCES = ["nf_api.hip", "nf_kernels.hip", "nf_narrow.hip", "nf_narrow64.hip", "nf_medium.hip",
           "nf_eval.hip", "nf_calib.hip", "nf_skinny.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    # no packed fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the library)")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"build step failed ({res.returncode}): {' '.join(cmd)}\n"
                           f"{res.stdout}\n{res.stderr}")


def build(verbose: bool = False) -> str:
    objdir = os.path.join(ROOT, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs = [os.path.join(objdir, os.path.splitext(src)[0] + ".o") for src in SOURCES]
    cmds = [[hipcc(), *HIPCC_FLAGS, "-c", "-I", os.path.join(ROOT, "include"), "-I", CSRC,
             os.path.join(CSRC, src), "-o", obj] for src, obj in zip(SOURCES, objs)]
    # one compiler process per source, at most as many as the CPUs this
    # process may use
    workers = max(1, min(len(cmds), len(os.sched_getaffinity(0)), 8))
    with concurrent.futures.ThreadPoolExecutor(workers) as pool:
        for f in [pool.submit(_run, c, verbose) for c in cmds]:
            f.result()
    rocm_lib = os.path.join(os.path.dirname(os.path.dirname(os.path.realpath(hipcc()))), "lib")
    tmp = LIB + ".tmp"
    _run([hipcc(), "-shared", "-fPIC", *objs, "-o", tmp, f"-Wl,-rpath,{rocm_lib}"], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
