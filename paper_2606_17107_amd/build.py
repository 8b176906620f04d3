"""Build libpkv.so (HIP, gfx950) in-tree: ``python -m paper_2606_17107_amd.build``.

Every ``csrc/*.hip`` file is compiled with hipcc for gfx950 into ``_build/``
and linked into ``paper_2606_17107_amd/libpkv.so``.  Packed-FP32 instruction
selection is disabled for all device code.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD_DIR = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libpkv.so")
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (need ROCm to build libpkv)")


def compile_flags():
    return [
        "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wall", "-Wno-unused-function", "-I", INCLUDE, "-I", CSRC,
    ]


# Per-source device-compiler options.  The MLA kernel's score MFMAs
# accumulate in VGPRs (its output accumulators, written only by inline
# assembly, take the whole AGPR file): the compiler chooses one register file
# for all MFMA builtins of a function.
FILE_FLAGS = {
    "attn_mla_bf16.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link libpkv.so; returns the library path."""
    os.makedirs(BUILD_DIR, exist_ok=True)
    cc = hipcc()
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    procs = []
    objs = []
    for src in srcs:
        obj = os.path.join(BUILD_DIR, os.path.basename(src) + ".o")
        objs.append(obj)
        cmd = [cc] + compile_flags() + FILE_FLAGS.get(os.path.basename(src), []) + ["-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    failed = []
    for src, p in procs:
        out, _ = p.communicate()
        text = out.decode(errors="replace")
        # hipcc's host pass does not know the packed-fp32 target feature; that warning is harmless.
        lines = [l for l in text.splitlines() if "packed-fp32-ops" not in l]
        if p.returncode != 0:
            failed.append(src)
            sys.stderr.write("\n".join(lines) + "\n")
        elif verbose and lines:
            print("\n".join(lines))
    if failed:
        raise RuntimeError("hipcc failed for: " + ", ".join(os.path.basename(f) for f in failed))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [cc, "--offload-arch=" + ARCH, "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    build_copy(verbose)
    return LIB


COPY_SRC = os.path.join(PKG, "probe", "stream_copy.hip")
COPY_LIB = os.path.join(PKG, "libpkv_copy.so")


def build_copy(verbose: bool = False) -> str:
    """The stream-copy reference kernel the benchmark times beside the splice (its own library)."""
    tmp = COPY_LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc()] + compile_flags() + ["-shared", COPY_SRC, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    out = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if out.returncode != 0:
        sys.stderr.write(out.stdout.decode(errors="replace"))
        raise RuntimeError("hipcc failed for " + COPY_SRC)
    os.replace(tmp, COPY_LIB)
    return COPY_LIB


if __name__ == "__main__":
    print(build(verbose=True))
