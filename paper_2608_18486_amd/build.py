"""Build libwhitematter.so for gfx950 with hipcc (in-tree, next to this file).

Usage: python -m paper_2608_18486_amd.build  (or call build()).
"""
from __future__ import annotations

import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libwhitematter.so")
# source -> extra flags. The projection GEMMs keep their accumulators in arch
# VGPRs (MFMA VGPR form): their epilogue reads the accumulators in place, where
# AGPR accumulators would be copied out all at once at the end of the K loop.
SOURCES = {
    "wm_api.hip": [],
    "wm_pool.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
    "wm_attend.hip": [],
    "wm_backward.hip": [],
    "wm_grad.hip": [],
    "wm_calib.hip": [],
}
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
OBJDIR = os.path.join(ROOT, "_build")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    # no packed-fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]
NOISE = "'-packed-fp32-ops' is not a recognized feature"


def _run(cmds, verbose):
    procs = []
    for cmd in cmds:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append(subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT,
                                      text=True))
    failed = []
    for cmd, p in zip(cmds, procs):
        out, _ = p.communicate()
        msgs = [ln for ln in out.splitlines() if NOISE not in ln]
        if p.returncode != 0:
            failed.append("\n".join(msgs))
        elif verbose and msgs:
            print("\n".join(msgs))
    if failed:
        raise RuntimeError("hipcc failed:\n" + "\n".join(failed))


def build(verbose: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    tag = "%d" % os.getpid()
    objs, cmds = [], []
    for src, extra in SOURCES.items():
        obj = os.path.join(OBJDIR, src.replace(".hip", ".%s.o" % tag))
        objs.append(obj)
        cmds.append([HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj])
    _run(cmds, verbose)
    tmp = LIB + ".tmp" + tag
    try:
        _run([[HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]], verbose)
    finally:
        for o in objs:
            if os.path.exists(o):
                os.remove(o)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
