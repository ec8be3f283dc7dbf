"""Build libattn.so (HIP kernels for gfx950 plus the C ABI) in-tree.

    python -m paper_2605_05023_amd.build               # libattn.so
    python -m paper_2605_05023_amd.build --lds-poison  # libattn_poison.so

Each translation unit is compiled to an object in parallel, then linked.
Packed fp32 instructions are disabled for all device code. The LDS-poisoning
debug build (ATTN_LDS_POISON, kernel_params.h) fills every kernel's LDS with
all-ones bytes first; tests compare it with the release build bit for bit.
"""
from __future__ import annotations

import concurrent.futures
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libattn.so")
LIB_POISON = os.path.join(PKG, "libattn_poison.so")
BUILD_DIR = os.path.join(PKG, "_build")
ARCH = "gfx950"

DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
COMMON = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
          "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-Wall", "-Wno-unused-function"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def sources():
    return sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                  if f.endswith((".hip", ".cpp")))


def _compile(src: str, poison: bool = False) -> str:
    bdir = BUILD_DIR + ("_poison" if poison else "")
    obj = os.path.join(bdir, os.path.basename(src) + ".o")
    extra = ["-DATTN_LDS_POISON=1"] if poison else []
    cmd = [hipcc(), *COMMON, *DEVICE_FLAGS, *extra, "-c", src, "-o", obj]
    res = subprocess.run(cmd, capture_output=True, text=True)
    # hipcc's host pass does not know the device-only feature flag; drop that note
    err = "\n".join(l for l in res.stderr.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{err}")
    if err.strip():
        sys.stderr.write(err + "\n")
    return obj


def build(verbose: bool = False, poison: bool = False) -> str:
    lib = LIB_POISON if poison else LIB
    os.makedirs(BUILD_DIR + ("_poison" if poison else ""), exist_ok=True)
    srcs = sources()
    with concurrent.futures.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
        objs = list(ex.map(lambda s: _compile(s, poison), srcs))
    tmp = lib + ".tmp"
    cmd = [hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build(verbose=True, poison="--lds-poison" in sys.argv[1:])
