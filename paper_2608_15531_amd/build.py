"""Build libfq.so in-tree: host C++ with g++, HIP kernels with hipcc for gfx950."""

from __future__ import annotations

import os
import shutil
import subprocess
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(HERE, "_build")
LIB_NAME = "libfq.so"
LIB_PATH = os.path.join(HERE, LIB_NAME)
# the streaming-read probe (a measurement reference, include/fq_probe.h) is a
# library of its own
PROBE_LIB_PATH = os.path.join(HERE, "libfqprobe.so")
PROBE_SOURCES = ["probe.hip"]
# the instrumented build (per-wave timestamps, include/fq_debug.h): the same
# sources with FQ_WAVE_STAMPS defined
STAMPS_LIB_PATH = os.path.join(HERE, "libfq_stamps.so")
# the bf16 GEMM comparator on hipBLASLt (include/fq_gemm_ref.h): host code
# only, a library of its own
GEMM_LIB_PATH = os.path.join(HERE, "libfqgemm.so")
GEMM_SOURCES = ["gemm_ref.cpp"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")

HOST_SOURCES = ["capi.cpp", "tilecoo.cpp", "quant.cpp"]
HIP_SOURCES = ["kernels.hip"]

# Packed-fp32 VALU forms are kept out of every HIP object.  MFMA results stay
# in ordinary VGPRs (the accumulation registers would need a copy-out per
# tile before the fp32 scale and zero-point step).  Kernel arguments are
# preloaded into scalar registers.
HIP_FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             "-mllvm", "-amdgpu-mfma-vgpr-form=1",
             # the hardware loads the first 14 kernel-argument dwords into
             # scalar registers before a wave starts (no argument fetch on the
             # path to a kernel's first loads)
             "-mllvm", "-amdgpu-kernarg-preload-count=14",
             "-Wall", "-Wno-unused-result"]
HOST_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra"]


def _hipcc() -> str:
    return os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        raise RuntimeError(f"command failed ({res.returncode}): {' '.join(cmd)}\n"
                           f"{res.stdout}\n{res.stderr}")
    return res


def build(verbose: bool = False) -> str:
    """Compile every source and link libfq.so, libfqprobe.so, the
    instrumented libfq_stamps.so and the comparator libfqgemm.so next to this
    file; returns the path of libfq.so."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    incs = ["-I", INCLUDE, "-I", CSRC]
    jobs = []
    for src in HOST_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".o")
        jobs.append(["g++", *HOST_FLAGS, *incs, "-c", os.path.join(CSRC, src), "-o", obj])
    for src in GEMM_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".o")
        jobs.append(["g++", *HOST_FLAGS, "-D__HIP_PLATFORM_AMD__", "-isystem",
                     os.path.join(ROCM, "include"), *incs, "-c", os.path.join(CSRC, src), "-o", obj])
    for src in HIP_SOURCES + PROBE_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".o")
        jobs.append([_hipcc(), *HIP_FLAGS, *incs, "-c", os.path.join(CSRC, src), "-o", obj])
    stamp_objs = []
    for src in HIP_SOURCES:
        obj = os.path.join(BUILD_DIR, src + ".stamps.o")
        stamp_objs.append(obj)
        jobs.append([_hipcc(), *HIP_FLAGS, "-DFQ_WAVE_STAMPS", *incs, "-c", os.path.join(CSRC, src),
                     "-o", obj])
    with ThreadPoolExecutor(max_workers=4) as ex:
        list(ex.map(lambda c: _run(c, verbose), jobs))
    objs = [j[-1] for j in jobs if j[-1] not in stamp_objs]
    probe_objs = [o for o in objs if os.path.basename(o)[:-2] in PROBE_SOURCES]
    gemm_objs = [o for o in objs if os.path.basename(o)[:-2] in GEMM_SOURCES]
    lib_objs = [o for o in objs if o not in probe_objs and o not in gemm_objs]
    host_objs = [o for o in lib_objs if os.path.basename(o)[:-2] in HOST_SOURCES]
    for path, ob in ((LIB_PATH, lib_objs), (PROBE_LIB_PATH, probe_objs),
                     (STAMPS_LIB_PATH, host_objs + stamp_objs)):
        tmp = path + ".tmp"
        _run([_hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *ob, "-o", tmp], verbose)
        shutil.move(tmp, path)
    rocm_lib = os.path.join(ROCM, "lib")
    _run(["g++", "-shared", "-fPIC", *gemm_objs, "-L", rocm_lib, "-lhipblaslt", "-lamdhip64",
          f"-Wl,-rpath,{rocm_lib}", "-o", GEMM_LIB_PATH + ".tmp"], verbose)
    shutil.move(GEMM_LIB_PATH + ".tmp", GEMM_LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
