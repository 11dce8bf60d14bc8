"""Build libmoe.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2607_01844_amd.build        # or __graft_entry__.build()
"""
from __future__ import annotations

import concurrent.futures as cf
import hashlib
import json
import os
import subprocess
import sys
import tempfile

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
OBJ = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libmoe.so")
# sha256 of each object's gfx950 machine code (.text of its device code
# object), written beside the library at every build: a stored measurement
# names the code it was taken on, and stays valid while that code is unchanged
DEVICE_TEXT = os.path.join(PKG, "libmoe.device_text.json")
SOURCES = ["api.hip", "route.hip", "route_bwd.hip", "permute.hip", "combine.hip", "gemm.hip",
           "chunked.hip", "vocab.hip", "llep.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
CFLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
    # packed fp32 instructions stay off on this target (see the design notes)
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result", "-Wno-unused-command-line-argument",
    "-I", os.path.join(ROOT, "include"), "-I", CSRC,
]


def _compile(src: str) -> str:
    obj = os.path.join(OBJ, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *CFLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines()
                    if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{out}")
    if out.strip():
        print(out, file=sys.stderr)
    return obj


LLVM = "/opt/rocm/llvm/bin"


def device_text_sha256(obj: str) -> str:
    """sha256 of the .text section of the gfx950 code object embedded in a
    hipcc object file (comments and host-only edits leave it unchanged), or
    None for an object without device code."""
    sections = subprocess.run([f"{LLVM}/llvm-readelf", "-S", obj], check=True,
                              capture_output=True, text=True).stdout
    if ".hip_fatbin" not in sections:
        return None
    with tempfile.TemporaryDirectory() as tmp:
        fat, co, text = (os.path.join(tmp, n) for n in ("fat.bin", "dev.co", "text.bin"))
        subprocess.run([f"{LLVM}/llvm-objcopy", "-O", "binary", "--only-section=.hip_fatbin", obj,
                        fat], check=True, capture_output=True)
        subprocess.run([f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o",
                        f"--input={fat}", f"--targets=hipv4-amdgcn-amd-amdhsa--{ARCH}",
                        f"--output={co}"], check=True, capture_output=True)
        subprocess.run([f"{LLVM}/llvm-objcopy", "-O", "binary", "--only-section=.text", co, text],
                       check=True, capture_output=True)
        with open(text, "rb") as fh:
            return hashlib.sha256(fh.read()).hexdigest()


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link libmoe.so (always rebuilds)."""
    os.makedirs(OBJ, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    hashes = {src: device_text_sha256(obj) for src, obj in zip(SOURCES, objs)}
    with open(DEVICE_TEXT + ".tmp", "w") as fh:
        json.dump(hashes, fh, indent=1, sort_keys=True)
    os.replace(DEVICE_TEXT + ".tmp", DEVICE_TEXT)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
