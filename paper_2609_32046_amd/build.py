"""Build ``libcacheback.so`` (the HIP kernels and the C ABI) for gfx950.

Run as ``python paper_2609_32046_amd/build.py`` (by path: importing the
package would load the library being rebuilt).  hipcc cross-compiles on a
host without a GPU.  The library is built in-tree, next to this file.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
SOURCES = ["api.hip", "score.hip", "score_bf16_d128.hip", "score_bf16_d64.hip",
           "score_f32_d128.hip", "score_f32_d64.hip", "score_pos_bf16_d128.hip",
           "score_pos_bf16_d64.hip", "score_pos_f32_d128.hip", "score_pos_f32_d64.hip",
           "select.hip", "compact.hip", "position.hip"]
LIB = os.path.join(HERE, "libcacheback.so")
ARCH = "gfx950"
FLAGS = [f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
         # packed-fp32 VALU forms are kept out of the generated code
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wall", "-Wno-unused-function"]


def hipcc() -> str:
    cand = os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc")
    return cand if os.path.exists(cand) else (shutil.which("hipcc") or "hipcc")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (res.stdout + res.stderr).splitlines()
                     if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{msgs}")
    if verbose and msgs.strip():
        print(msgs)


def build(verbose: bool = False, extra=()) -> str:
    """Compile every source to an object (in parallel), then link the library."""
    objdir = tempfile.mkdtemp(prefix="cb_build_")
    try:
        objs = [os.path.join(objdir, s.replace(".hip", ".o")) for s in SOURCES]
        jobs = min(len(SOURCES), max(1, os.cpu_count() or 1))
        with concurrent.futures.ThreadPoolExecutor(jobs) as pool:
            futs = [pool.submit(_run, [hipcc(), *FLAGS, "-c", os.path.join(CSRC, s), "-o", o,
                                       *extra], verbose)
                    for s, o in zip(SOURCES, objs)]
            for f in futs:
                f.result()
        _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", LIB + ".tmp",
              *extra], verbose)
        os.replace(LIB + ".tmp", LIB)
    finally:
        shutil.rmtree(objdir, ignore_errors=True)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
