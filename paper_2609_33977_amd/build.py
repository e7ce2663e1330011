"""Build libgroupmask.so (gfx950 HIP kernels + C-ABI layer) in-tree with hipcc.

Usage: python paper_2609_33977_amd/build.py   (or build() from Python)
"""
from __future__ import annotations

import concurrent.futures
import os
import re
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OBJ = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libgroupmask.so")
ARCH = "gfx950"

SOURCES = ["gate.hip", "budget.hip", "index.hip", "gemv.hip", "gemm.hip", "distill.hip", "hyper.hip", "abi.cpp"]

# Packed fp32 VALU ops are kept out of the generated code; the host pass
# warns that it does not know the feature, which is harmless.
COMMON = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    "-Wall", "-Werror", "-Wno-unused-command-line-argument",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


# The GEMM kernels issue their MFMAs through inline assembly with the
# accumulators as tied operands the register allocator cannot see through: if
# it ever moved one (spilling, or copying between the two register files near
# the register limit) the results would be silently wrong.  Every kernel's
# resource report is therefore checked at build time: no kernel may use
# scratch memory or spill vector registers, and the kernels with tied
# accumulators (sources that include gm_gemm.h) must stay at least 8 registers
# below the 256 that two waves per SIMD allow (variants at 252-256 gave wrong
# results).
TIED_ACC_SOURCES = ("gemm.hip", "distill.hip")
TIED_ACC_MAX_REGS = 248
_REMARK = re.compile(r"remark:\s+(Function Name|VGPRs|AGPRs|ScratchSize \[bytes/lane\]|VGPRs Spill):\s*(\S+)")


def _resource_report(src: str, stderr: str):
    """Per kernel: its VGPRs, AGPRs, scratch bytes per lane and spilled VGPRs, from clang's remarks."""
    kernels, cur = {}, None
    for key, val in _REMARK.findall(stderr):
        if key == "Function Name":
            cur = kernels.setdefault(val, {})
        elif cur is not None:
            cur[key] = int(val)
    problems = []
    for name, r in kernels.items():
        if r.get("ScratchSize [bytes/lane]", 0) or r.get("VGPRs Spill", 0):
            problems.append(f"{src}: {name} uses scratch or spills vector registers: {r}")
        regs = r.get("VGPRs", 0) + r.get("AGPRs", 0)
        if src in TIED_ACC_SOURCES and regs > TIED_ACC_MAX_REGS:
            problems.append(f"{src}: {name} uses {regs} registers (> {TIED_ACC_MAX_REGS}) with tied accumulators")
    return kernels, problems


def _hipcc() -> str:
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the ROCm toolchain is required to build libgroupmask")


def _compile(src: str) -> str:
    out = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    cmd = [_hipcc(), *COMMON, "-Rpass-analysis=kernel-resource-usage", "-c", os.path.join(CSRC, src), "-o", out]
    if src.endswith(".cpp"):
        cmd[1:1] = ["-x", "hip"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
    _, problems = _resource_report(src, r.stderr)
    if problems:
        os.remove(out)
        raise RuntimeError("kernel resource check failed:\n" + "\n".join(problems))
    return out


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link the shared library; returns its path."""
    os.makedirs(OBJ, exist_ok=True)
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


def build_host_sanitized(out_dir: str) -> str:
    """A copy of the library whose host code (the C-ABI layer: validation, layouts,
    dispatch) is built with AddressSanitizer and UndefinedBehaviorSanitizer; the
    device code is unchanged.  Needs the objects of a normal build.  Load it with
    GM_LIBRARY_PATH and the clang ASan runtime preloaded."""
    os.makedirs(out_dir, exist_ok=True)
    obj = os.path.join(out_dir, "abi_san.o")
    cmd = [_hipcc(), "-x", "hip", f"--offload-arch={ARCH}", "-O1", "-g", "-std=c++17", "-fPIC",
           "-fvisibility=hidden", "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-omit-frame-pointer", "-c", os.path.join(CSRC, "abi.cpp"), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitizer compile failed:\n{r.stderr}")
    others = [os.path.join(OBJ, os.path.splitext(src)[0] + ".o") for src in SOURCES if src != "abi.cpp"]
    missing = [o for o in others if not os.path.exists(o)]
    if missing:
        raise FileNotFoundError(f"build the library first: {missing}")
    lib = os.path.join(out_dir, "libgroupmask_san.so")
    clangxx = os.path.join(os.path.dirname(os.path.realpath(_hipcc())), "..", "llvm", "bin", "clang++")
    if not os.path.exists(clangxx):
        clangxx = "/opt/rocm/llvm/bin/clang++"
    link = [clangxx, "-shared", "-fPIC", "-shared-libsan", "-fsanitize=address,undefined", "-o", lib, obj, *others,
            "-L/opt/rocm/lib", "-lamdhip64"]
    r = subprocess.run(link, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"sanitizer link failed:\n{r.stderr}")
    return lib


def asan_runtime() -> str:
    """Path of the clang AddressSanitizer runtime that a sanitized build needs preloaded."""
    import glob
    found = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not found:
        raise FileNotFoundError("clang ASan runtime not found")
    return found[-1]


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
