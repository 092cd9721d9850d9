"""Build libmarche.so (the C-ABI HIP library) for gfx950 with hipcc.

Every call compiles from source: each translation unit to an object in
``_build/`` (in parallel), then one shared library next to this file.

    python -m paper_2506_12035_amd.build
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor
from typing import Optional

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmarche.so")
SOURCES = ("marche_api.cpp", "marche_noalloc.hip", "k_elementwise.hip", "k_gemm.hip",
           "k_attn.hip", "k_select.hip", "k_mar.hip")
ARCH = "gfx950"

# -packed-fp32-ops: keep the compiler from forming packed fp32 VALU ops.
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-Wall", "-Wno-unused-function"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libmarche.so)")


# Per-source device flags.  The attention kernels hold only a few dozen
# accumulators per lane, and MFMA results in the AGPR file would cost a copy
# to and from the VGPRs for every softmax step on them, so their MFMAs take
# and produce VGPRs.  The GEMM tiles keep the compiler's choice (256
# accumulators per lane live in the AGPRs).
EXTRA = {"k_attn.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    lang = [] if src.endswith(".cpp") else ["-x", "hip"]
    cmd = [hipcc(), *COMMON, *EXTRA.get(src, []), *lang, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", "-Wl,--no-undefined", *objs,
           "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


# Host-side sources of the C ABI (argument validation, workspace layout,
# launch sequence); the sanitized build instruments these for the host only.
HOST_SOURCES = ("marche_api.cpp", "marche_noalloc.hip")
SAN_LIB = os.path.join(BUILD, "libmarche_san.so")
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
             "-Xarch_host", "-fno-omit-frame-pointer", "-Xarch_host", "-fno-sanitize-recover=all"]


def asan_runtime() -> Optional[str]:
    """The clang AddressSanitizer runtime matching hipcc's host compiler."""
    import glob
    hits = sorted(glob.glob("/opt/rocm/lib/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    return hits[-1] if hits else None


def build_sanitized() -> str:
    """libmarche_san.so: the host-side sources built with AddressSanitizer and
    UndefinedBehaviorSanitizer (host code only; device code is untouched),
    linked with the kernel objects of the last build().  For running the
    host-only ABI tests under the sanitizers; the runtime is preloaded by the
    caller (asan_runtime())."""
    os.makedirs(BUILD, exist_ok=True)
    objs = []
    for src in SOURCES:
        obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
        if src in HOST_SOURCES:
            obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".san.o")
            lang = [] if src.endswith(".cpp") else ["-x", "hip"]
            cmd = [hipcc(), *COMMON, *SAN_FLAGS, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
            r = subprocess.run(cmd, capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
        elif not os.path.exists(obj):
            _compile(src)
        objs.append(obj)
    tmp = SAN_LIB + ".tmp"
    cmd = [hipcc(), "-shared", "-fPIC", f"--offload-arch={ARCH}", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, SAN_LIB)
    return SAN_LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
