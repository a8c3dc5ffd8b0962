"""Build libreco.so (the gfx950 HIP kernels and the C ABI) in-tree with hipcc.

Usage: ``python -m paper_2608_04771_amd.build`` or ``build_library()``.
Always recompiles; the objects go to ``paper_2608_04771_amd/_build/`` and the
library to ``paper_2608_04771_amd/libreco.so``.  ``build_c_driver()`` then
compiles ``tests/c_abi/reco_c_driver``, a plain C client of the ABI."""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libreco.so")
ARCH = "gfx950"

HIP_SOURCES = ["decode_attn.hip", "score.hip", "select_compact.hip", "pool_scores.hip", "logits.hip"]
HOST_SOURCES = ["abi.cpp", "decode_plan.cpp"]

# Packed fp32 instructions are kept out of every kernel (v_pk_* fp32 forms).
NO_PACKED_FP32 = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the HIP library cannot be built")


def _run(cmd):
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # The host pass does not know the packed-fp32 feature and says so; drop that noise.
    out = "\n".join(l for l in res.stdout.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build_library(verbose: bool = False) -> str:
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    common = ["-O3", "-std=c++17", "-fPIC", "-Wall", f"-I{os.path.join(ROOT, 'include')}"]
    jobs = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        jobs.append((obj, [hipcc, "-x", "hip", f"--offload-arch={ARCH}", *common, *NO_PACKED_FP32,
                           "-c", os.path.join(CSRC, src), "-o", obj]))
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD, src + ".o")
        # fp64 host policies are computed without contraction, as the formulas are written
        jobs.append((obj, [hipcc, f"--offload-arch={ARCH}", *common, "-ffp-contract=off", "-c",
                           os.path.join(CSRC, src), "-o", obj]))
    with cf.ThreadPoolExecutor(max_workers=min(8, len(jobs))) as ex:
        outs = list(ex.map(lambda j: _run(j[1]), jobs))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    tmp = LIB + ".tmp"
    _run([hipcc, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *[j[0] for j in jobs]])
    os.replace(tmp, LIB)
    return LIB


C_DRIVER_SRC = os.path.join(ROOT, "tests", "c_abi", "reco_c_driver.c")
C_DRIVER = os.path.join(ROOT, "tests", "c_abi", "reco_c_driver")


def build_c_driver() -> str:
    """Compile the plain C11 client of the ABI (a GPU test runs it) against the
    built libreco.so and the HIP runtime, with gcc: no HIP device code in it."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        raise RuntimeError("no C compiler found for the C ABI client")
    tmp = C_DRIVER + ".tmp"
    _run([cc, "-std=c11", "-O2", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
          f"-I{os.path.join(rocm, 'include')}", f"-I{os.path.join(ROOT, 'include')}", C_DRIVER_SRC, "-o", tmp,
          f"-L{PKG}", "-lreco", f"-L{os.path.join(rocm, 'lib')}", "-lamdhip64",
          "-Wl,-rpath,$ORIGIN/../../paper_2608_04771_amd", f"-Wl,-rpath,{os.path.join(rocm, 'lib')}"])
    os.replace(tmp, C_DRIVER)
    return C_DRIVER


if __name__ == "__main__":
    path = build_library(verbose="-v" in sys.argv)
    print(path)
    print(build_c_driver())
