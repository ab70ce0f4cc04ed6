"""Build ``libmebp.so`` (the C-ABI library) for gfx950 with hipcc, in-tree.

Usage: ``python -m paper_2510_03425_amd.build`` or ``build()`` from Python.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libmebp.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
SOURCES = ["api.hip", "gemm_q4.hip", "gemm_big.hip", "attention.hip", "elementwise.hip", "lora.hip", "optim.hip", "timing.hip"]
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function",
    # no packed fp32 VALU ops (v_pk_*_f32) in generated code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


# Variants: "" is the product library. "asan" instruments the host code (argument
# validation, workspace layout, launch orchestration) with AddressSanitizer; the device
# code is built as usual. It is loaded with the sanitizer runtime preloaded (see
# asan_runtime()) by the host-only tests in a subprocess.
VARIANTS = {"": [], "asan": ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]}


def lib_path(variant: str = "") -> str:
    # test-only variants stay in the build folder, beside their objects
    return LIB if not variant else os.path.join(BUILD, f"libmebp_{variant}.so")


def asan_runtime() -> str:
    """Path of the AddressSanitizer runtime of the ROCm clang that builds the library."""
    import glob
    hits = sorted(glob.glob("/opt/rocm/llvm/lib/clang/*/lib/linux/libclang_rt.asan-x86_64.so"))
    if not hits:
        raise RuntimeError("no libclang_rt.asan-x86_64.so under /opt/rocm/llvm")
    return hits[-1]


def _compile(src: str, variant: str = "") -> str:
    obj = os.path.join(BUILD, (variant + "_" if variant else "") + src.replace(".hip", ".o"))
    cmd = [HIPCC, *FLAGS, *VARIANTS[variant], "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in ln]
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n" + "\n".join(msgs))
    if msgs:
        sys.stderr.write("\n".join(msgs) + "\n")
    return obj


def build(verbose: bool = False, variant: str = "") -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = min(len(SOURCES), max(1, min(8, os.cpu_count() or 1)))
    with ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(lambda src: _compile(src, variant), SOURCES))
    out = lib_path(variant)
    tmp = out + ".tmp"
    cmd = [HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", *VARIANTS[variant], *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, out)
    if verbose:
        print("built", out)
    return out


if __name__ == "__main__":
    build(verbose=True, variant=sys.argv[1] if len(sys.argv) > 1 else "")
