"""Build librlk.so (HIP for gfx950) in-tree with hipcc.

Usage: python -m paper_2608_16798_amd.build   (or call build()).
Every call recompiles; objects go to paper_2608_16798_amd/_build/.
RLK_EXTRA_FLAGS (environment) appends hipcc flags, e.g. "-DRLK_KS=64 -DRLK_NSTAGE=4" for the GEMM
pipeline geometry.

Host sanitizers: python -m paper_2608_16798_amd.build --host-sanitizers builds librlk_hostsan.so,
whose host code (argument validation, workspace layout, the chunk plan, the prefix-tree packer)
is compiled with AddressSanitizer and UndefinedBehaviorSanitizer (device code unchanged), then
runs the host-only tests against it with the ASan runtime preloaded (no GPU needed).
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


# Host-only sanitizer flags: -Xarch_host keeps them off the device code.
SAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined", "-Xarch_host",
             "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
SAN_OBJ = os.path.join(PKG, "_build_hostsan")
SAN_LIB = os.path.join(PKG, "librlk_hostsan.so")


def _compile(src: str, sanitize: bool = False) -> str:
    obj = os.path.join(SAN_OBJ if sanitize else OBJ, os.path.basename(src)[:-4] + ".o")
    check = os.path.basename(src) in NO_SCRATCH and not sanitize
    cmd = [HIPCC, *CFLAGS, *(SAN_FLAGS if sanitize else []), *([_REMARK] if check else []), "-c", src, "-o", obj]
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


def build(verbose: bool = True, sanitize: bool = False) -> str:
    lib = SAN_LIB if sanitize else LIB
    os.makedirs(SAN_OBJ if sanitize else OBJ, exist_ok=True)
    srcs = _sources()
    with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda src: _compile(src, sanitize), srcs))
    tmp = lib + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *(["-Xarch_host", "-shared-libsan"] if sanitize else []),
           "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}", file=sys.stderr)
    return lib


HOST_TESTS = ["tests/test_abi.py", "tests/test_tree_pack.py", "tests/test_binding_args.py"]


def run_host_sanitizers() -> int:
    """Build librlk_hostsan.so and run the host-only tests against it under ASan + UBSan."""
    lib = build(sanitize=True)
    rt = subprocess.run([HIPCC.replace("hipcc", "amdclang++") if os.path.exists(HIPCC.replace("hipcc", "amdclang++"))
                         else "clang++", "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True,
                        text=True).stdout.strip()
    if not rt or not os.path.exists(rt):
        rt = os.path.join(os.path.dirname(os.path.realpath(HIPCC)), "..", "llvm", "lib", "clang")
        cands = [os.path.join(dp, f) for dp, _, fs in os.walk(rt) for f in fs if f == "libclang_rt.asan-x86_64.so"]
        rt = cands[0] if cands else ""
    if not rt:
        raise RuntimeError("AddressSanitizer runtime libclang_rt.asan-x86_64.so not found")
    env = dict(os.environ, LD_PRELOAD=rt, RLK_LIBRARY=lib,
               ASAN_OPTIONS="detect_leaks=0:abort_on_error=1:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    root = os.path.dirname(PKG)
    print(f"host sanitizers: {lib} with {rt}", file=sys.stderr)
    return subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider", *HOST_TESTS], cwd=root,
                          env=env).returncode


if __name__ == "__main__":
    if "--host-sanitizers" in sys.argv[1:]:
        sys.exit(run_host_sanitizers())
    build()
