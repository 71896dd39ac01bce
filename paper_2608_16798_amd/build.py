"""Build librlk.so (HIP for gfx950) in-tree with hipcc.

Usage: python -m paper_2608_16798_amd.build   (or call build()).
Every call recompiles; objects go to paper_2608_16798_amd/_build/.
RLK_EXTRA_FLAGS (environment) appends hipcc flags, e.g. "-DRLK_KS=64 -DRLK_NSTAGE=4" for the GEMM
pipeline geometry.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "librlk.so")
ARCH = os.environ.get("RLK_OFFLOAD_ARCH", "gfx950")

HIPCC = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
# Packed fp32 VALU forms are disabled for all device code.
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
CFLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-Wall", "-Wno-unused-function",
          "-Wno-unused-variable"] + DEVICE_FLAGS + os.environ.get("RLK_EXTRA_FLAGS", "").split()


def _sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".hip"))


# The GEMM kernels are laid out to fit the register file: a spill to scratch memory would put
# vector-memory traffic into the main loop, so it fails the build instead.
NO_SCRATCH = {"k_gemm.hip"}
_REMARK = "-Rpass-analysis=kernel-resource-usage"


def _scratch_users(text: str):
    name, bad = None, []
    for line in text.splitlines():
        if "Function Name:" in line:
            name = line.split("Function Name:")[1].split()[0]
        elif "ScratchSize [bytes/lane]:" in line:
            if int(line.split("ScratchSize [bytes/lane]:")[1].split()[0]) != 0:
                bad.append(name)
    return bad


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.basename(src)[:-4] + ".o")
    check = os.path.basename(src) in NO_SCRATCH
    cmd = [HIPCC, *CFLAGS, *([_REMARK] if check else []), "-c", src, "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = r.stdout + r.stderr
    keep, in_remark = [], False
    for line in out.splitlines():
        if _REMARK in line:
            in_remark = True  # the remark and its source-context lines
            continue
        if in_remark and (line.strip().startswith("|") or line.split("|")[0].strip().isdigit()):
            continue
        in_remark = False
        if "packed-fp32-ops" not in line:
            keep.append(line)
    msgs = "\n".join(keep)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{msgs}")
    if check and _scratch_users(out):
        raise RuntimeError(f"{src}: kernels use scratch memory: {_scratch_users(out)}")
    if msgs.strip():
        print(msgs, file=sys.stderr)
    return obj


def build(verbose: bool = True) -> str:
    os.makedirs(OBJ, exist_ok=True)
    srcs = _sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(_compile, srcs))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}", file=sys.stderr)
    return LIB


if __name__ == "__main__":
    build()
