"""Build libisoquant.so in-tree: HIP kernels for gfx950 plus host C++.

    python paper_2603_28430_amd/build.py

(run as a script, or loaded by file path: importing the package itself loads
the library this script produces).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libisoquant.so")
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

# Device code: gfx950 only; packed-FP32 VALU instructions are disabled; matrix
# instructions read and write ordinary VGPRs (their results feed VALU code
# directly, without accumulation-register copies and the waits they need).
DEVICE_FLAGS = ["-x", "hip", f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
                "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                "-mllvm", "-amdgpu-mfma-vgpr-form",
                "-Wall", "-Wno-unused-parameter"]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include",
              "-Wall", "-Wextra", "-Wno-unused-parameter"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        sys.stderr.write(r.stdout + r.stderr)
        raise RuntimeError("build step failed: " + " ".join(cmd))
    return r


def build(verbose: bool = False) -> str:
    obj_dir = os.path.join(PKG, "_build")
    os.makedirs(obj_dir, exist_ok=True)
    inc = [f"-I{INCLUDE}", f"-I{CSRC}"]
    jobs = []
    for src in ("isoq_kernels.hip", "isoq_kernels_8d.hip", "isoq_kernels_m.hip", "isoq_scores.hip",
                "isoq_scores_8d.hip", "isoq_scores_qjl.hip", "isoq_qjl.hip", "isoq_generic_full.hip", "isoq_generic_fast.hip",
                "isoq_generic_2d.hip", "isoq_generic_8d.hip", "isoq_qjl_append.hip", "isoq_packed.hip",
                "isoq_packed_8d.hip", "isoq_packed_qjl.hip", "isoq_scores_generic.hip"):
        jobs.append([HIPCC, *DEVICE_FLAGS, *inc, "-c", os.path.join(CSRC, src), "-o",
                     os.path.join(obj_dir, src + ".o")])
    for src in ("isoq_api.cpp", "isoq_host_params.cpp"):
        jobs.append([os.path.join(ROCM, "llvm", "bin", "clang++"), *HOST_FLAGS, *inc, "-c",
                     os.path.join(CSRC, src), "-o", os.path.join(obj_dir, src + ".o")])
    with cf.ThreadPoolExecutor(max_workers=len(jobs)) as ex:
        for r in ex.map(_run, jobs):
            if verbose and (r.stdout or r.stderr):
                sys.stderr.write(r.stdout + r.stderr)
    objs = [j[-1] for j in jobs]
    tmp = LIB + ".tmp"
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp,
          f"-L{ROCM}/lib", "-lamdhip64"])
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
