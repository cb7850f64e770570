"""Builds libprhs.so (HIP for gfx950) in-tree with hipcc.

    python -m paper_2602_08329_amd.build [-v]
    python -m paper_2602_08329_amd.build --host-sanitize OUT.so

Every source is recompiled on each call; objects go to ``_build/`` next to
this file and the shared library to ``paper_2602_08329_amd/libprhs.so``.
With --host-sanitize the host code (argument validation, workspace sizing,
dispatch) is built with AddressSanitizer and UndefinedBehaviorSanitizer into
OUT.so (objects beside it) for CPU-side checks; device code is built as usual
and is not instrumented.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libprhs.so")
SOURCES = ["prhs_api.hip", "select.hip", "dilate.hip", "attention.hip", "gate.hip", "prefill.hip"]

ARCH = "gfx950"
FLAGS = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
    # no packed fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-function", "-Wno-unused-variable",
]


# Per-source flags.  prefill.hip: MFMA accumulators in ordinary VGPRs; with
# the online-softmax rescale of the accumulators in its loop, the default
# (accumulation registers) costs register copies on every key tile.
EXTRA_FLAGS = {"prefill.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}


def hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the HIP library cannot be built")
    return path


# Host-side sanitizers (each flag applies to the host compilation only).
SANITIZE = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-omit-frame-pointer", "-g"]


def build(verbose: bool = False, host_sanitize: str = None) -> str:
    out_lib = LIB if host_sanitize is None else os.path.abspath(host_sanitize)
    objdir = BUILD if host_sanitize is None else out_lib + ".objs"
    os.makedirs(objdir, exist_ok=True)
    cc = hipcc()
    flags = list(FLAGS)
    link_extra = []
    if host_sanitize is not None:
        flags = [f if f != "-O3" else "-O1" for f in flags] + SANITIZE
        link_extra = SANITIZE[:4]
    procs = []
    objs = []
    for src in SOURCES:
        obj = os.path.join(objdir, src.replace(".hip", ".o"))
        objs.append(obj)
        cmd = [cc, *flags, *EXTRA_FLAGS.get(src, []), "-I", INCLUDE, "-I", CSRC, "-c",
               os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                                            text=True)))
    errors = []
    for src, p in procs:
        out, _ = p.communicate()
        lines = [ln for ln in out.splitlines() if "packed-fp32-ops" not in ln]
        if p.returncode != 0:
            errors.append(f"--- {src}\n" + "\n".join(lines))
        elif verbose and lines:
            print("\n".join(lines))
    if errors:
        raise RuntimeError("hipcc failed:\n" + "\n".join(errors))
    tmp = out_lib + ".tmp"
    cmd = [cc, "-shared", "-fPIC", f"--offload-arch={ARCH}", *link_extra, *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout)
    os.replace(tmp, out_lib)
    return out_lib


if __name__ == "__main__":
    san = None
    if "--host-sanitize" in sys.argv:
        san = sys.argv[sys.argv.index("--host-sanitize") + 1]
    print(build(verbose="-v" in sys.argv, host_sanitize=san))
