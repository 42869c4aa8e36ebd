"""Build librefadapt.so (gfx950) in-tree with hipcc.

Usage: python -m paper_2609_32415_amd.csrc.build   (or call ``build()``)

Every source is compiled for gfx950 only. Packed fp32 VALU instructions are
disabled (``-packed-fp32-ops``) for all device code.
"""

from __future__ import annotations

import hashlib
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
PKG = os.path.dirname(HERE)
ROOT = os.path.dirname(PKG)
SOURCES = ["api.hip", "attn_bf16.hip", "attn_f32.hip", "stats.hip", "diag.hip", "probe.hip"]
LIB_NAME = "librefadapt.so"
ARCH = "gfx950"


def hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the ROCm toolchain is required to build librefadapt")
    return path


# Code-generation flags of every source (no paths: they also key the profiles' build hash).
CODEGEN_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-Wall",
    "-Wno-unused-function",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    # MFMA accumulators in ordinary vector registers: the softmax reads the
    # score tiles directly instead of copying them out of AGPRs every tile.
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    # The scheduler's register-pressure tracking that spills fewer scalar registers to
    # vector lanes in the attention loop (80 instead of 109; about -0.5% launch time).
    "-mllvm", "-amdgpu-use-amdgpu-trackers=1",
]


def compile_flags():
    return [*CODEGEN_FLAGS, "-I", os.path.join(ROOT, "include")]


def kernel_build_sha256():
    """sha256 over the bf16 attention source and CODEGEN_FLAGS: the key under which the
    profiles/ summaries record the build they were measured on."""
    h = hashlib.sha256(open(os.path.join(HERE, "attn_bf16.hip"), "rb").read())
    h.update("\0".join(CODEGEN_FLAGS).encode())
    return h.hexdigest()


def build(verbose=False, jobs=4):
    """Compile every source to an object under _build/ and link the shared library."""
    out_dir = os.path.join(ROOT, "_build")
    os.makedirs(out_dir, exist_ok=True)
    cc = hipcc()
    procs = []
    objs = []
    for src in SOURCES:
        obj = os.path.join(out_dir, src.replace(".hip", ".o"))
        objs.append(obj)
        cmd = [cc, *compile_flags(), "-c", os.path.join(HERE, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
        if len(procs) >= jobs:
            _drain(procs)
    _drain(procs)
    lib = os.path.join(PKG, LIB_NAME)
    tmp = lib + ".tmp"
    cmd = [cc, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}")
    os.replace(tmp, lib)
    build_example(verbose)
    return lib


def build_example(verbose=False):
    """Compile examples/joint_attn_c.c, a plain-C caller of the library (C99, the HIP runtime
    API and include/refadapt.h only), next to its source; it finds the library through its
    run path."""
    src = os.path.join(PKG, "examples", "joint_attn_c.c")
    exe = os.path.join(PKG, "examples", "joint_attn_c")
    rocm = os.path.dirname(os.path.dirname(os.path.realpath(hipcc())))
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        raise RuntimeError("no C compiler found for the C example")
    cmd = [cc, "-std=c99", "-O2", "-Wall", "-Wextra", "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(rocm, "include"), src, "-L", PKG, "-lrefadapt", "-L", os.path.join(rocm, "lib"),
           "-lamdhip64", "-lm", "-Wl,-rpath,$ORIGIN/..", "-Wl,-rpath," + os.path.join(rocm, "lib"), "-o", exe + ".tmp"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"C example build failed:\n{r.stdout}")
    os.replace(exe + ".tmp", exe)
    return exe


def _drain(procs):
    errors = []
    while procs:
        src, p = procs.pop(0)
        out, _ = p.communicate()
        if p.returncode != 0:
            errors.append(f"{src}:\n{out}")
        elif out.strip():
            print(f"[{src}]\n{out}", file=sys.stderr)
    if errors:
        raise RuntimeError("compilation failed:\n" + "\n".join(errors))


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
