"""Build libduet.so in-tree: HIP sources for gfx950 with hipcc, host C++ with g++."""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OBJDIR = os.path.join(ROOT, "_build", "obj")
LIB = os.path.join(PKG, "libduet.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ROCM_LIB = "/opt/rocm/lib"
ARCH = "gfx950"
HIP_FLAGS = ["--offload-arch=" + ARCH, "-O3", "-fPIC", "-std=c++17", "-Wall",
             # no packed-fp32 instructions anywhere in the device code
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             # atomics stay as written: the decode kernel's one-lane counter atomic must not get the
             # wave-aggregation rewrite, which reads its result right after issue
             "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
             "-I" + INCLUDE, "-I" + CSRC]
# MFMA accumulators in VGPRs: the online-softmax rescale works on them in place.
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form"]


def _hip_flags(src):
    return HIP_FLAGS + VGPR_FORM


CXX_FLAGS = ["-O2", "-fPIC", "-std=c++17", "-Wall", "-I" + INCLUDE, "-I" + CSRC,
             "-I/opt/rocm/include", "-D__HIP_PLATFORM_AMD__"]


def _run(cmd):
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"build failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return r


def build(verbose: bool = False, out: str = LIB, extra=(), objdir: str = OBJDIR) -> str:
    """Compile every source and link libduet.so (always recompiles).  `extra` adds hipcc flags
    to every HIP source; `out` and `objdir` place the result elsewhere."""
    os.makedirs(objdir, exist_ok=True)
    jobs = []
    for src in sorted(glob.glob(os.path.join(CSRC, "*.hip"))):
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        jobs.append([HIPCC, *_hip_flags(src), *extra, "-c", src, "-o", obj])
    for src in sorted(glob.glob(os.path.join(CSRC, "*.cpp"))):
        obj = os.path.join(objdir, os.path.basename(src) + ".o")
        jobs.append([shutil.which("g++") or "g++", *CXX_FLAGS, "-c", src, "-o", obj])
    workers = max(1, min(len(jobs), 8))
    with cf.ThreadPoolExecutor(workers) as ex:
        for r in ex.map(_run, jobs):
            if verbose and r.stderr:
                print(r.stderr)
    objs = [j[-1] for j in jobs]
    tmp = out + ".tmp"
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp, *objs, "-L" + ROCM_LIB, "-lhipblaslt",
          "-Wl,-rpath," + ROCM_LIB])
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True))
