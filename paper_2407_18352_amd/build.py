"""Build ``libhpacml.so`` (HIP kernels for gfx950 + the C ABI) in-tree.

Usage: ``python -m paper_2407_18352_amd.build`` (or ``build()`` from Python).
Objects go to ``_build/``; the library lands next to this file.
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
OUT = os.path.join(PKG, "libhpacml.so")
BUILD = os.path.join(ROOT, "_build")
ARCH = "gfx950"


def _hipcc() -> str:
    for c in (os.path.join(os.environ.get("ROCM_PATH", "/opt/rocm"), "bin", "hipcc"), shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wno-unused-function", "-I", INCLUDE, "-I", CSRC]
# packed fp32 VALU forms are kept out of the generated code on purpose
DEVICE = ["-x", "hip", "--offload-arch=" + ARCH, "-Xclang", "-target-feature", "-Xclang",
          "-packed-fp32-ops"]


# the register-resident bf16 kernel keeps its activations in accumulation
# registers as MFMA B operands; results and C operands go to vector registers
PER_FILE = {f: ["-mllvm", "-amdgpu-mfma-vgpr-form"]
            for f in ("mlp_bf16r.hip", "mlp_bf16r_h256_nh1.hip", "mlp_bf16r_h256_nh2.hip", "mlp_bf16r_h256_nh3.hip")}


def build(verbose: bool = False) -> str:
    hipcc = _hipcc()
    os.makedirs(BUILD, exist_ok=True)
    jobs = []
    for src in sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.cpp"))):
        obj = os.path.join(BUILD, os.path.basename(src) + ".o")
        cmd = [hipcc] + COMMON + (DEVICE if src.endswith(".hip") else ["-x", "c++"]) + PER_FILE.get(os.path.basename(src), [])
        cmd += ["-c", src, "-o", obj]
        jobs.append((cmd, obj, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)))
    objs = []
    failed = []
    for cmd, obj, proc in jobs:
        out, _ = proc.communicate()
        text = out.decode(errors="replace")
        # the host pass does not know the packed-fp32 device feature; harmless
        text = "\n".join(l for l in text.splitlines() if "packed-fp32-ops" not in l)
        if proc.returncode != 0:
            failed.append((" ".join(cmd), text))
        elif verbose and text.strip():
            print(text)
        objs.append(obj)
    if failed:
        for c, t in failed:
            sys.stderr.write("FAILED: %s\n%s\n" % (c, t))
        raise RuntimeError("HIP build failed")
    tmp = OUT + ".tmp%d" % os.getpid()
    # hipBLASLt: the per-layer matmuls of the layer-by-layer path
    link = [hipcc, "-shared", "-fPIC", "--hip-link", "--offload-arch=" + ARCH] + objs + ["-lhipblaslt", "-o", tmp]
    res = subprocess.run(link, stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if res.returncode != 0:
        sys.stderr.write(res.stdout.decode(errors="replace"))
        raise RuntimeError("link failed")
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose=True))
