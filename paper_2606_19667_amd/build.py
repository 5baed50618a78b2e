"""Builds libcw.so in-tree for gfx950.

    python -m paper_2606_19667_amd.build [-v] [--sanitize]

The host sources build with g++, the HIP sources with hipcc for gfx950; hipcc
links the shared library against the HIP runtime.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys
import tempfile

try:
    from . import asm_check
except ImportError:   # run as a script
    import asm_check

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libcw.so")

ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

HOST_SOURCES = ["cw_host.cpp", "cw_tree.cpp", "cw_proj.cpp"]
HIP_SOURCES = ["cw_kernels.hip", "cw_qkv.hip", "cw_probe.hip"]

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-mcode-object-version=5",
    # no NaN operands reach the kernels' float code (masked scores are -inf,
    # never NaN), which lets max reductions use v_max3 without quieting
    "-fno-honor-nans",
    # keep the compiler from forming packed fp32 VALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
]
HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-Wall", "-Wextra"]
# Per-source extra flags. The attention kernel's step has uniform (wave-wide)
# branches only; structurizing them makes the register allocator keep two
# copies of the 64-register output accumulator across the branch arms, which
# overflows the 256-register budget of two waves per SIMD.
EXTRA_FLAGS = {"cw_kernels.hip": ["-mllvm", "-structurizecfg-skip-uniform-regions=true"]}


def _run(cmd):
    proc = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if proc.returncode != 0:
        raise RuntimeError("build step failed:\n" + " ".join(cmd) + "\n" + proc.stdout)
    return proc.stdout


# Host sources built with AddressSanitizer and UndefinedBehaviorSanitizer
# (`--sanitize`): the library is linked by g++ into libcw_sanitized.so, which
# cw.py loads when CW_LIBRARY names it (the process preloads libasan/libubsan).
SANITIZE_FLAGS = ["-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                  "-fno-sanitize-recover=undefined"]
LIB_SANITIZED = os.path.join(PKG, "libcw_sanitized.so")


def build(verbose: bool = False, sanitize: bool = False) -> str:
    """Compiles every source and links libcw.so (libcw_sanitized.so with
    `sanitize`); returns its path."""
    incs = [f"-I{INCLUDE}", f"-I{CSRC}"]
    gxx = shutil.which("g++") or "g++"
    host_flags = HOST_FLAGS + (SANITIZE_FLAGS if sanitize else [])
    with tempfile.TemporaryDirectory(prefix="cw_build_") as tmp:
        objs = []
        for src in HOST_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            out = _run([gxx, *host_flags, *incs, "-c",
                        os.path.join(CSRC, src), "-o", obj])
            objs.append(obj)
            if verbose and out:
                print(out)
        for src in HIP_SOURCES:
            obj = os.path.join(tmp, src + ".o")
            out = _run([HIPCC, *HIP_FLAGS, *EXTRA_FLAGS.get(src, []), *incs, "-c", os.path.join(CSRC, src), "-o", obj])
            objs.append(obj)
            if verbose and out:
                print(out)
        # The attention kernel's untracked loads are checked on its assembly
        # (asm_check): no path may touch their registers before a covering wait.
        asm = os.path.join(tmp, "cw_kernels.s")
        _run([HIPCC, *HIP_FLAGS, *EXTRA_FLAGS["cw_kernels.hip"], *incs, "--cuda-device-only", "-S",
              os.path.join(CSRC, "cw_kernels.hip"), "-o", asm])
        with open(asm) as fh:
            report = asm_check.check(fh.read())
        if verbose:
            print("untracked loads checked:", report)
        tmp_lib = os.path.join(tmp, "libcw.so")
        if sanitize:
            rocm_lib = os.path.join(ROCM, "lib")
            _run([gxx, "-shared", "-fPIC", "-fsanitize=address,undefined", *objs, f"-L{rocm_lib}",
                  "-lamdhip64", f"-Wl,-rpath,{rocm_lib}", "-o", tmp_lib])
            shutil.move(tmp_lib, LIB_SANITIZED)
            return LIB_SANITIZED
        _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp_lib])
        shutil.move(tmp_lib, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, sanitize="--sanitize" in sys.argv))
