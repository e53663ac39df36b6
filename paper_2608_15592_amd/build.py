"""Build libestp.so from the HIP sources for gfx950 (MI355X).

Usage: ``python -m paper_2608_15592_amd.build`` (or ``__graft_entry__.build()``).
The library is written next to this file so it travels with the source tree.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libestp.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-fvisibility=hidden",
    "-shared",
    "-Wall",
    "-Wno-unused-command-line-argument",
    # keep the compiler from forming packed fp32 ALU instructions
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found")


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


# Host code only, AddressSanitizer: every -fsanitize flag sits behind -Xarch_host, so the gfx950
# device code is built exactly as in the plain library.  The runtime is linked dynamically; a
# process that loads this library (Python included) needs it preloaded: see asan_runtime().
ASAN_FLAGS = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fno-omit-frame-pointer",
              "-Xarch_host", "-shared-libsan", "-Xarch_host", "-g"]
ASAN_LIB = os.path.join(HERE, "libestp_asan.so")


def asan_runtime() -> str:
    """Path of the AddressSanitizer runtime that hipcc's clang links against."""
    res = subprocess.run([hipcc(), "-print-file-name=libclang_rt.asan-x86_64.so"], capture_output=True, text=True)
    path = res.stdout.strip()
    if res.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError("AddressSanitizer runtime not found")
    return path


def build(verbose: bool = False, out: str = LIB, defines=(), sanitize: bool = False) -> str:
    """Compile every HIP source into one shared library; returns its path.  ``sanitize`` adds
    AddressSanitizer to the host code (default output libestp_asan.so)."""
    if sanitize and out == LIB:
        out = ASAN_LIB
    tmp = out + ".tmp"
    cmd = [hipcc(), *HIPCC_FLAGS, *(ASAN_FLAGS if sanitize else []), *[f"-D{d}" for d in defines], f"-I{INCLUDE}",
           f"-I{CSRC}", *sources(), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode}")
    os.replace(tmp, out)
    return out


if __name__ == "__main__":
    print(build(verbose=True, sanitize=os.environ.get("ASAN") == "1"))
