"""Builds libsra.so (HIP for gfx950 + host scheduler) in-tree with hipcc.

    python -m paper_2606_13872_amd.build      # or: python paper_2606_13872_amd/build.py
Every call recompiles. Objects go to paper_2606_13872_amd/_build/, the library next to
this file.
"""
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
LIB = os.path.join(PKG, "libsra.so")

SOURCES = ["schedule.cpp", "sra_api.cpp", "sra_fwd.hip", "sra_bwd.hip", "sra_dq.hip", "sra_dkv.hip",
           "sra_compact.hip", "sra_noalloc.hip"]

COMMON = [
    "-O3", "-std=c++17", "-fPIC", "-Wall",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]
# Device code only for gfx950. Packed-FP32 instructions are disabled in device code.
HIP_FLAGS = ["-x", "hip", "--offload-arch=gfx950", "-Xclang", "-target-feature",
             "-Xclang", "-packed-fp32-ops"]
# The dK/dV and dQ kernels select their compiler-visible MFMAs in VGPR form: their AGPRs hold
# the gradient sums (written by inline-assembly MFMAs), and S/dP must stay in VGPRs next to them.
_VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]
EXTRA_FLAGS = {"sra_dkv.hip": _VGPR_FORM, "sra_dq.hip": _VGPR_FORM}
COMPILE_TIMEOUT_S = 900


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the ROCm toolchain is required to build libsra")
    return path


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    path = os.path.join(CSRC, src)
    if src.endswith(".hip"):
        cmd = [hipcc(), *HIP_FLAGS, *EXTRA_FLAGS.get(src, []), *COMMON, "-c", path, "-o", obj]
    else:  # host-only C++ (the scheduler includes no HIP header)
        cmd = [hipcc(), *COMMON, "-c", path, "-o", obj] if src == "sra_api.cpp" else \
              ["g++", *COMMON, "-c", path, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True, timeout=COMPILE_TIMEOUT_S)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=6) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", "--offload-arch=gfx950", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


# Host-only build for the sanitizer run: the scheduler and the C ABI compiled with g++ under
# AddressSanitizer and UndefinedBehaviorSanitizer, the kernel launchers replaced by stubs that
# report hipErrorNotSupported. No device code is built. The tests of the schedules and of the
# ABI's host validation load it through SRA_HOST_LIB, with libasan preloaded into Python:
#   python -m paper_2606_13872_amd.build --sanitize
#   SRA_HOST_LIB=paper_2606_13872_amd/_build/sanitize/libsra_host.so \
#   LD_PRELOAD=$(g++ -print-file-name=libasan.so) ASAN_OPTIONS=detect_leaks=0 \
#   UBSAN_OPTIONS=halt_on_error=1:print_stacktrace=1 python -m pytest tests/test_schedule.py tests/test_abi.py
SAN_DIR = os.path.join(BUILD, "sanitize")
SAN_LIB = os.path.join(SAN_DIR, "libsra_host.so")
SAN_SOURCES = ["schedule.cpp", "sra_api.cpp", "sra_host_stubs.cpp"]
SAN_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined", "-fno-omit-frame-pointer", "-g",
             "-O1"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def build_sanitized(verbose: bool = False) -> str:
    os.makedirs(SAN_DIR, exist_ok=True)
    # g++ 11 has no __bf16; the host code only passes bf16 tensors around as pointers
    hip = ["-D__HIP_PLATFORM_AMD__", "-D__bf16=uint16_t", "-I", os.path.join(ROCM, "include")]
    flags = [f for f in COMMON if f != "-O3"]
    objs = []
    for src in SAN_SOURCES:
        obj = os.path.join(SAN_DIR, os.path.splitext(src)[0] + ".o")
        cmd = ["g++", *flags, *hip, *SAN_FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True, timeout=COMPILE_TIMEOUT_S)
        if r.returncode != 0:
            raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
        objs.append(obj)
    cmd = ["g++", "-shared", *SAN_FLAGS, "-o", SAN_LIB, *objs, "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
           f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    if verbose:
        print("built", SAN_LIB)
    return SAN_LIB


if __name__ == "__main__":
    if "--sanitize" in sys.argv[1:]:
        build_sanitized(verbose=True)
    else:
        build(verbose=True)
    sys.exit(0)
