"""Build libspecctx.so (HIP kernels + C ABI) for gfx950 with hipcc.

    python -m paper_2512_00722_amd.build

Objects are compiled in parallel into _build/ next to this file and linked
into paper_2512_00722_amd/libspecctx.so (in-tree, so it travels with the
source tree).  Every call recompiles.
"""

from __future__ import annotations

import concurrent.futures
import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
ROOT = os.path.dirname(PKG)
LIB = os.path.join(PKG, "libspecctx.so")
BUILD_DIR = os.path.join(PKG, "_build")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-fvisibility=hidden",
    "-Wall",
    "-Wno-unused-result",
    # packed fp32 instructions stay disabled in every HIP translation unit
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    f"-I{os.path.join(ROOT, 'include')}",
]


# Per-source additions.  mla.hip: MFMA results in VGPRs rather than AGPRs.
# The MLA attention's latent accumulators are also rescaled by the vector
# ALU, rarely; held in AGPRs, the compiler copies every one of them into
# VGPRs on each chunk for that branch and spills the queries.  In VGPRs, the
# queries (only ever MFMA operands) take the AGPRs instead.
EXTRA_FLAGS = {"mla.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def flags_for(src: str) -> list:
    return FLAGS + EXTRA_FLAGS.get(os.path.basename(src), [])


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp")))


def _compile(src: str) -> str:
    obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
    cmd = [HIPCC, *flags_for(src), "-x", "hip", "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD_DIR, exist_ok=True)
    srcs = sources()
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB} from {len(srcs)} sources")
    return LIB


SANITIZED_LIB = os.path.join(BUILD_DIR, "libspecctx_hostsan.so")


def build_sanitized(verbose: bool = False) -> str:
    """A host-sanitizer variant for the CPU ABI tests: the C-ABI host code
    (spec_api.cpp: validation, workspace carve-up, dispatch) compiled by g++
    with AddressSanitizer and UndefinedBehaviorSanitizer, linked with the
    kernel objects of the last build().  No device code is instrumented.
    Loading it needs the ASan runtime preloaded (LD_PRELOAD)."""
    objs = [os.path.join(BUILD_DIR, os.path.basename(s) + ".o") for s in sources()
            if not s.endswith("spec_api.cpp")]
    if not all(os.path.exists(o) for o in objs):
        build(verbose)
    san_obj = os.path.join(BUILD_DIR, "spec_api.hostsan.o")
    gxx = os.environ.get("CXX", "g++")
    rocm = os.path.dirname(os.path.dirname(HIPCC))
    cmd = [gxx, "-std=c++17", "-O1", "-g", "-fPIC", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-D__HIP_PLATFORM_AMD__", f"-I{os.path.join(rocm, 'include')}",
           f"-I{os.path.join(ROOT, 'include')}", "-c", os.path.join(CSRC, "spec_api.cpp"),
           "-o", san_obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized compile failed:\n{' '.join(cmd)}\n{r.stderr}")
    tmp = SANITIZED_LIB + ".tmp"
    cmd = [gxx, "-shared", "-fPIC", "-fsanitize=address,undefined", "-o", tmp, san_obj, *objs,
           f"-L{os.path.join(rocm, 'lib')}", "-lamdhip64", f"-Wl,-rpath,{os.path.join(rocm, 'lib')}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitized link failed:\n{' '.join(cmd)}\n{r.stderr}")
    os.replace(tmp, SANITIZED_LIB)
    if verbose:
        print(f"built {SANITIZED_LIB} (host ASan + UBSan on the C-ABI layer)")
    return SANITIZED_LIB


def clean():
    shutil.rmtree(BUILD_DIR, ignore_errors=True)
    if os.path.exists(LIB):
        os.remove(LIB)


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
