"""Build ``libsl.so`` (the gfx950 HIP kernels plus the C ABI) in-tree with hipcc.

Every call compiles from scratch; the library lands next to this file.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIBRARY = os.path.join(HERE, "libsl.so")
SOURCES = ["decode_split.hip", "decode_shared.hip", "merge.hip", "append.hip", "engine.hip", "api.cpp",
           "engine.cpp", "dispatch.cpp", "noalloc.hip"]
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-result",
    "-mcode-object-version=5",
    # no packed-fp32 instructions anywhere (the hardware forms are avoided on purpose)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary VGPRs: the online softmax rescales them with
    # vector ALU instructions, which cannot read accumulation registers
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    "-I", os.path.join(ROOT, "include"),
]


def _hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def build(output: str = LIBRARY, extra: list[str] | None = None, verbose: bool = False,
          objdir: str | None = None) -> str:
    """Compile every source and link ``output``; returns its path."""
    objdir = objdir or os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    flags = HIPCC_FLAGS + list(extra or [])

    def compile_one(src: str) -> str:
        obj = os.path.join(objdir, src + ".o")
        lang = ["-x", "hip"] if src.endswith(".hip") else []
        cmd = [_hipcc(), *flags, *lang, "-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.run(cmd, check=True)
        return obj

    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(compile_one, SOURCES))
    tmp = output + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, output)
    return output


# The whole library with its host code (the C ABI, the engine's host loop, dispatching)
# under the sanitizers and its GPU code unchanged: every flag applies to the host pass only.
HOST_SANITIZE_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                       "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
                       "-Xarch_host", "-g"]


# UBSan alone, for runs that use the GPU: ROCm's ASan runtime intercepts the HSA allocator for
# device-side checking, which cannot run here, so a process that touches the GPU takes no ASan.
HOST_UBSAN_FLAGS = ["-Xarch_host", "-fsanitize=undefined", "-Xarch_host", "-fno-sanitize=vptr",
                    "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-g"]


def clang_runtime(name: str) -> str | None:
    """A sanitizer runtime of the compiler hipcc drives (``asan`` or ``ubsan_standalone``), to
    preload into an uninstrumented Python."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    hits = sorted(glob.glob(os.path.join(rocm, "llvm", "lib", "clang", "*", "lib", "linux",
                                         f"libclang_rt.{name}-x86_64.so")))
    return hits[-1] if hits else None


# Host-only build of the dispatching code (csrc/dispatch.cpp, no GPU code) with the host
# sanitizers, loaded through SL_DISPATCH_LIBRARY by the sanitizer test.
SANITIZE_FLAGS = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g"]


def build_dispatch_host(output: str, extra: list[str] | None = None) -> str:
    """Compile csrc/dispatch.cpp alone with the host C++ compiler into the shared library
    ``output`` (the HIP headers are only read for the status type)."""
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    cmd = ["g++", "-std=c++17", "-O1", "-fPIC", "-shared", "-Wall", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(rocm, "include"), "-I", os.path.join(ROOT, "include"), *(extra or []),
           os.path.join(CSRC, "dispatch.cpp"), "-o", output]
    subprocess.run(cmd, check=True)
    return output


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
