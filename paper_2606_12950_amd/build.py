"""Build libmaestro.so (gfx950) in-tree with hipcc, and beside it libmaestro_calibrate.so, the
measurement-only matrix-core ceiling kernel that bench.py --mfma-ceiling times.

Usage: python -m paper_2606_12950_amd.build [-v]
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libmaestro.so")
SOURCES = ("api.hip", "predict.hip", "roles.hip", "route.hip", "fitness.hip", "prioritize.hip")
CALIBRATE_LIB = os.path.join(PKG, "libmaestro_calibrate.so")
CALIBRATE_SOURCE = "calibrate.hip"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    # exact, unfused float arithmetic: route scores and latency quantisation are bit-exact
    # contracts, so no multiply-add contraction anywhere in the library
    "-ffp-contract=off",
    # never emit packed-FP32 instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fvisibility=hidden",
    "-Wall", "-Wno-unused-function",
    f"-I{INCLUDE}", f"-I{CSRC}",
]
# per-source additions: the predictor converts its MFMA accumulators with vector ALU
# instructions, which read only architectural VGPRs; keeping MFMA results there avoids a copy
# out of the accumulation registers for every converted value
EXTRA = {"predict.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _compile(src: str, outdir: str, verbose: bool) -> str:
    obj = os.path.join(outdir, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                     if "packed-fp32-ops" not in l and l.strip())
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{msgs}")
    if verbose and msgs:
        print(msgs, flush=True)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every HIP source for gfx950 and link libmaestro.so next to this file."""
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    with tempfile.TemporaryDirectory(prefix="maestro_build_") as tmp:
        with ThreadPoolExecutor(max_workers=len(SOURCES) + 1) as ex:
            objs = list(ex.map(lambda s: _compile(s, tmp, verbose), SOURCES + (CALIBRATE_SOURCE,)))
        for lib, lib_objs in ((LIB, objs[:-1]), (CALIBRATE_LIB, objs[-1:])):
            out = os.path.join(tmp, os.path.basename(lib))
            cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *lib_objs, "-o", out]
            if verbose:
                print(" ".join(cmd), flush=True)
            subprocess.run(cmd, check=True)
            shutil.copyfile(out, lib + ".tmp")
            os.replace(lib + ".tmp", lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
