"""Build libmot.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2607_28979_amd.build

Every kernel source compiles with packed fp32 instructions disabled
(-packed-fp32-ops), and the objects link into csrc/libmot.so.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
ROOT = os.path.dirname(HERE)
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(CSRC, "libmot.so")
# (source, object name, preprocessor definitions); the fused kernel's
# instantiation file is compiled once per (d_in, d_out) so they build in parallel
SOURCES = [(f, os.path.splitext(f)[0], {}) for f in
           ("mot_api.hip", "k_router.hip", "k_routed.hip", "k_f32.hip", "k_f32_mfma.hip", "k_bf16_unfused.hip", "k_bf16_gemm256.hip",
            "k_bf16_fused.hip", "k_project.hip", "k_replay.hip", "k_backbone.hip")]
SOURCES += [("k_bf16_fused_inst.hip", "k_bf16_fused_%d_%d" % (a, b),
             {"MOT_FUSED_D_IN": a, "MOT_FUSED_D_OUT": b})
            for a in (128, 256, 512) for b in (128, 256, 512)]
# per-source device-compiler options: these kernels keep their MFMA
# accumulators in VGPRs (the attention softmax rescales them in place and the
# GEMM epilogues read them; the AGPR form copies them in and out)
_VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form"]
EXTRA = {f: _VGPR_FORM for f in ("k_replay.hip", "k_backbone.hip", "k_project.hip", "k_bf16_unfused.hip")}


def hipcc() -> str:
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found (ROCm is required to build libmot)")


def flags():
    return ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wno-unused-command-line-argument",
            "-I", os.path.join(ROOT, "include")]


def _compile(entry) -> str:
    src, name, defs = entry
    obj = os.path.join(BUILD, name + ".o")
    cmd = [hipcc(), *flags(), *EXTRA.get(src, []), *["-D%s=%s" % kv for kv in defs.items()], "-c", os.path.join(CSRC, src),
           "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("compile failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    jobs = min(len(SOURCES), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(jobs) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed: %s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr))
    os.replace(tmp, LIB)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
    sys.exit(0)
