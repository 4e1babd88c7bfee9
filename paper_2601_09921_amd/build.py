"""Builds the HIP library libpwdec.so in-tree for gfx950 with hipcc."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libpwdec.so")
SOURCES = ["tok.hip", "attn.hip", "resident.hip", "readout.hip", "f32_window.hip", "stream.hip", "pwdec.cpp"]
# Per-source extra flags. The attention kernel keeps its MFMA accumulators in VGPRs (it needs
# far fewer than 256), so no copies between accumulation and arithmetic registers; the token
# kernel needs the AGPRs as accumulators.
EXTRA_FLAGS = {"attn.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "--offload-arch=gfx950", "-fPIC",
    "-Wall", "-Wno-unused-function",
    # no packed-fp32 VALU instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build the decoder library)")


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    return subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)


def _finish(proc):
    out, _ = proc.communicate()
    noise = "is not a recognized feature for this target"
    msgs = [ln for ln in out.splitlines() if noise not in ln]
    if proc.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    return msgs


def build(verbose: bool = False) -> str:
    """Compile every source (in parallel) and link libpwdec.so; always recompiles."""
    objdir = os.path.join(HERE, "_build")
    os.makedirs(objdir, exist_ok=True)
    objs, procs = [], []
    for src in SOURCES:
        obj = os.path.join(objdir, src + ".o")
        objs.append(obj)
        cmd = [hipcc(), *HIPCC_FLAGS, *EXTRA_FLAGS.get(src, []), "-x", "hip", "-c",
               os.path.join(CSRC, src), "-o", obj]
        procs.append(_run(cmd, verbose))
    msgs = []
    for p in procs:
        msgs += _finish(p)
    tmp = LIB + ".tmp"
    msgs += _finish(_run([hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", *objs, "-o", tmp], verbose))
    if verbose and msgs:
        print("\n".join(msgs), file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


def build_host_asan(verbose: bool = False) -> str:
    """The library with the host code of pwdec.cpp (configuration checks, blob parser, handle
    logic) instrumented by AddressSanitizer and the device code unchanged, linked from the
    kernels' objects of build() into _build/libpwdec_asan.so for the host checks in
    tests/asan. Builds the kernels' objects first if they are missing."""
    objdir = os.path.join(HERE, "_build")
    kernels = [os.path.join(objdir, src + ".o") for src in SOURCES if src != "pwdec.cpp"]
    if not all(os.path.exists(o) for o in kernels):
        build(verbose)
    obj = os.path.join(objdir, "pwdec.cpp.asan.o")
    sanitize = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer"]
    _finish(_run([hipcc(), *HIPCC_FLAGS, *sanitize, "-x", "hip", "-c", os.path.join(CSRC, "pwdec.cpp"), "-o", obj],
                 verbose))
    out = os.path.join(objdir, "libpwdec_asan.so")
    rocm_lib = os.path.join(os.path.dirname(os.path.dirname(hipcc())), "lib")
    link = ["g++", "-shared", "-fsanitize=address", *kernels, obj, f"-L{rocm_lib}", "-lamdhip64",
            f"-Wl,-rpath,{rocm_lib}", "-o", out]
    _finish(_run(link, verbose))
    return out


if __name__ == "__main__":
    print(build(verbose=True))
