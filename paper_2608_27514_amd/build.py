"""Builds libtrajspec.so (gfx950) in-tree with hipcc.

Usage: python -m paper_2608_27514_amd.build  [--verbose]
"""

import os
import shutil
import subprocess
import sys

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
CSRC = os.path.join(PKG_DIR, "csrc")
LIB_NAME = "libtrajspec.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)
# measurement aid: the streaming-read floor of the logit pass (not part of the C ABI)
FLOOR_PATH = os.path.join(PKG_DIR, "libtrajfloor.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    "-shared",
    "-Wall",
    "-Wno-unused-function",
    # never let the compiler form packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
]


def hipcc_path():
    for cand in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libtrajspec)")


def sources():
    return [os.path.join(CSRC, "trajspec.hip")]


def source_digest():
    """sha256 (hex) over every file the library is built from (the kernel sources under csrc/,
    the C ABI header) and the compiler flags; stamped into traj_version() at build time so that
    a loaded binary can be checked against the checked-out sources."""
    import hashlib
    h = hashlib.sha256()
    files = [os.path.join(CSRC, f) for f in sorted(os.listdir(CSRC)) if f.endswith((".hpp", ".h"))]
    files += sources()
    files.append(os.path.join(ROOT, "include", "traj_spec.h"))
    for path in files:
        h.update(os.path.relpath(path, ROOT).encode() + b"\0")
        with open(path, "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    h.update(" ".join(HIPCC_FLAGS).encode())
    return h.hexdigest()


def build(verbose=False, extra_flags=()):
    """Compile the library; always rebuilds.  Returns the library path."""
    tmp = LIB_PATH + ".tmp"
    stamp = f'-DTRAJ_SOURCE_DIGEST="{source_digest()}"'
    cmd = [hipcc_path(), *HIPCC_FLAGS, *extra_flags, stamp, "-I", os.path.join(ROOT, "include"), *sources(), "-o",
           tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(line for line in (res.stdout + res.stderr).splitlines()
                    if "packed-fp32-ops" not in line)
    if res.returncode != 0:
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{out}")
    if verbose and out.strip():
        print(out, flush=True)
    os.replace(tmp, LIB_PATH)
    build_floor(verbose)
    return LIB_PATH


def build_floor(verbose=False):
    """Compile libtrajfloor.so, the logit pass's streaming-read floor (a measurement aid)."""
    tmp = FLOOR_PATH + ".tmp"
    cmd = [hipcc_path(), *HIPCC_FLAGS, "-I", CSRC, os.path.join(CSRC, "stream_floor.hip"), "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        out = "\n".join(line for line in (res.stdout + res.stderr).splitlines() if "packed-fp32-ops" not in line)
        raise RuntimeError(f"hipcc failed ({res.returncode}):\n{out}")
    os.replace(tmp, FLOOR_PATH)
    return FLOOR_PATH


if __name__ == "__main__":
    print(build(verbose="--verbose" in sys.argv))
