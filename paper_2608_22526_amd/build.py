"""Builds the rs3 HIP library (gfx950) in place: paper_2608_22526_amd/librs3.so.

Usage: python -m paper_2608_22526_amd.build [-j N]
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OBJDIR = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "librs3.so")
SOURCES = ["host_check.cpp", "select.hip", "commit.hip", "readout.hip", "attend.hip", "rope.hip", "keepset.hip", "post.hip", "fused.hip", "stack.hip", "api.hip", "profile.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
# The attention kernel keeps its MFMA accumulators in arch VGPRs, so the
# online-softmax rescale is plain VALU work instead of AGPR round trips.
PER_FILE = {"readout.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"], "fused.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"]}
FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
    "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
    # packed fp32 VALU ops are kept off the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l)
    if p.returncode != 0:
        raise RuntimeError("command failed: %s\n%s" % (" ".join(cmd), out))
    return out


def build(jobs: int = 4, verbose: bool = False) -> str:
    os.makedirs(OBJDIR, exist_ok=True)
    objs = [os.path.join(OBJDIR, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    cmds = [[HIPCC] + FLAGS + PER_FILE.get(s, []) + ["-c", os.path.join(CSRC, s), "-o", o]
            for s, o in zip(SOURCES, objs)]
    with ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        outs = list(ex.map(_run, cmds))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    j = 4
    if "-j" in sys.argv:
        j = int(sys.argv[sys.argv.index("-j") + 1])
    print(build(j, verbose=True))
