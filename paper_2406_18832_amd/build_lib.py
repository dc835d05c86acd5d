"""Builds libot.so (all HIP sources under csrc/) in place, for gfx950 only.

Flags:
  -ffp-contract=off  the method's roundings are specified step by step; a
                     fused multiply-add would skip one of them.
  -Xclang -target-feature -Xclang -packed-fp32-ops
                     keep the compiler from emitting packed fp32 arithmetic.

build(sanitize=True) builds a copy whose host code (the C ABI's checks,
launch plans and dispatch) runs under AddressSanitizer and
UndefinedBehaviorSanitizer; the GPU code is built as usual.  Load it into a
process with the sanitizer runtime preloaded (asan_runtime() names it) and
the binding pointed at it (OT_LIBRARY).
"""
from __future__ import annotations

import glob
import hashlib
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libot.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared", f"--offload-arch={ARCH}",
    "-ffp-contract=off", "-fno-fast-math",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


# host side only: each sanitizer flag applies to the host pass alone
SANITIZE_FLAGS = [
    "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
    "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host", "-fno-omit-frame-pointer",
    "-g",
]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libot)")


def sources():
    return sorted(glob.glob(os.path.join(CSRC, "*.hip")))


def source_digest() -> str:
    """SHA-256 over what the library is built from: every csrc/*.hip and
    csrc/*.h and include/ot.h (each as its path relative to the repository,
    a zero byte and its contents, in path order), then the release compiler
    flags (HIPCC_FLAGS; a sanitizer build records the same digest).
    build() compiles it into the library, which ot_build_info() reports, so
    a loaded library can be matched against the sources in the tree."""
    root = os.path.dirname(HERE)
    files = sorted(glob.glob(os.path.join(CSRC, "*.hip")) + glob.glob(os.path.join(CSRC, "*.h")) +
                   [os.path.join(root, "include", "ot.h")])
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.relpath(f, root).encode() + b"\0")
        with open(f, "rb") as fh:
            h.update(fh.read())
    h.update(" ".join(HIPCC_FLAGS).encode())
    return h.hexdigest()


def asan_runtime() -> str:
    """Path of the compiler's AddressSanitizer runtime (to preload into a
    process that loads the sanitized library)."""
    clang = os.path.join(os.path.dirname(os.path.realpath(hipcc())), "..", "llvm", "bin", "clang")
    if not os.path.exists(clang):
        clang = "/opt/rocm/llvm/bin/clang"
    out = subprocess.run([clang, "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True)
    path = out.stdout.strip()
    if out.returncode != 0 or not os.path.isabs(path) or not os.path.exists(path):
        raise RuntimeError("AddressSanitizer runtime not found")
    return path


def build(verbose: bool = False, extra_flags=(), sanitize: bool = False, out: str = None) -> str:
    """Compiles every csrc/*.hip into libot.so next to this file (or into
    out) and returns its path.  Always recompiles.  sanitize=True: host code
    under AddressSanitizer and UndefinedBehaviorSanitizer."""
    lib = out or LIB
    tmp = lib + ".tmp"
    flags = list(HIPCC_FLAGS)
    if sanitize:
        flags = [f for f in flags if f != "-O3"] + ["-O1", *SANITIZE_FLAGS]
    cmd = [hipcc(), *flags, *extra_flags, f'-DOT_SOURCES_SHA256="{source_digest()}"', *sources(),
           "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode}")
    # hipcc's host pass does not know the packed-fp32 target feature and says
    # so; everything else it prints is shown
    noise = "packed-fp32-ops' is not a recognized feature"
    for line in (res.stdout + res.stderr).splitlines():
        if noise not in line and "warning: feature flag" not in line and line.strip():
            if verbose:
                print(line)
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose=True))
