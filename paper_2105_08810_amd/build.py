"""Build libsnn.so (the HIP kernels and their C ABI) for gfx950 with hipcc, in-tree.

    python -m paper_2105_08810_amd.build

Each .hip file compiles to its own object under csrc/_build/ (in parallel), then the objects
link into paper_2105_08810_amd/libsnn.so. hipcc cross-compiles, so no GPU is needed to build.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OBJDIR = os.path.join(CSRC, "_build")
LIB = os.path.join(PKG, "libsnn.so")

SOURCES = [
    "runtime.hip",
    "active_compact.hip",
    "lif_forward.hip",
    "sparse_backward.hip",
    "dw_mfma.hip",
    "dense_backward.hip",
    "readout_ce.hip",
    "train_step.hip",
    "conv_layer.hip",
]
# The forward and the compaction decide spikes and active sets, which must be bit-exact:
# no contraction of a*b+c into fused multiply-adds there.
EXACT = {"lif_forward.hip", "active_compact.hip"}

ARCH = os.environ.get("SNN_OFFLOAD_ARCH", "gfx950")
COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # packed fp32 VALU ops stay off (they are generated from plain float code otherwise)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-command-line-argument",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libsnn)")


def _compile(src: str) -> str:
    obj = os.path.join(OBJDIR, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc(), *COMMON, "-c", os.path.join(CSRC, src), "-o", obj]
    if src in EXACT:
        cmd.insert(1, "-ffp-contract=off")
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed on {src}:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    cmd = [hipcc(), "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


SAN_DIR = os.path.join(OBJDIR, "san")
SAN_LIB = os.path.join(SAN_DIR, "libsnn_san.so")
# AddressSanitizer and UndefinedBehaviorSanitizer on the host code only (argument validation,
# workspace sizing, planning); each -fsanitize= goes to the host pass alone
SAN_HOST = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]


def asan_runtime() -> str:
    """Path of the compiler's shared AddressSanitizer runtime (preloaded into a Python process
    that loads the sanitized library)."""
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    r = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    return r.stdout.strip()


def build_sanitized() -> str:
    """libsnn_san.so: the same sources with the host sanitizers (-O1 -g), for CPU tests of the
    argument validation. The device code is built as usual (it does not run in those tests)."""
    os.makedirs(SAN_DIR, exist_ok=True)
    flags = [f for f in COMMON if f != "-O3"] + ["-O1", "-g"] + SAN_HOST

    def one(src):
        obj = os.path.join(SAN_DIR, os.path.splitext(src)[0] + ".o")
        cmd = [hipcc(), *flags, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{' '.join(cmd)}\n{r.stderr}")
        return obj

    with ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(one, SOURCES))
    cmd = [hipcc(), "-shared", f"--offload-arch={ARCH}", *SAN_HOST, "-shared-libasan", "-o", SAN_LIB, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{' '.join(cmd)}\n{r.stderr}")
    return SAN_LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
