"""Build libcachescout.so in-tree with hipcc for gfx950.

    python -m paper_2608_14624_amd.build

compiles every ``csrc/*.hip`` source (and the host-only ``csrc/*.cpp``) into
``paper_2608_14624_amd/libcachescout.so``.
"""

import glob
import hashlib
import os
import shutil
import subprocess
import sys
import tempfile

PKG_DIR = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG_DIR)
LIB_NAME = "libcachescout.so"
LIB_PATH = os.path.join(PKG_DIR, LIB_NAME)
ARCH = "gfx950"


def hipcc():
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found; the HIP toolchain is required to build libcachescout.so")
    return path


def cxx():
    path = shutil.which("g++") or shutil.which("c++")
    if not path:
        raise RuntimeError("no host C++ compiler (g++) found")
    return path


def run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"{os.path.basename(cmd[0])} failed with exit code {res.returncode}")


def source_files():
    """Every file the library is built from: the sources and headers under
    csrc/ and the public header(s) under include/."""
    files = []
    for pattern in ("*.hip", "*.cpp", "*.h"):
        files += glob.glob(os.path.join(PKG_DIR, "csrc", pattern))
    files += glob.glob(os.path.join(ROOT, "include", "*.h"))
    return sorted(files)


def source_digest():
    """First 16 hex digits of a SHA-256 over the names and bytes of
    source_files(); the build embeds it in the library (cs_source_digest)."""
    h = hashlib.sha256()
    for path in source_files():
        h.update(os.path.relpath(path, ROOT).encode())
        h.update(b"\0")
        with open(path, "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    return h.hexdigest()[:16]


def build(verbose=False):
    """Compile the HIP sources and the host-only C++ into the shared library
    and return its path."""
    sources = sorted(glob.glob(os.path.join(PKG_DIR, "csrc", "*.hip")))
    host_sources = sorted(glob.glob(os.path.join(PKG_DIR, "csrc", "*.cpp")))
    includes = ["-I", os.path.join(ROOT, "include"), "-I", os.path.join(PKG_DIR, "csrc")]
    digest = f'-DCS_SOURCE_DIGEST="{source_digest()}"'

    tmp = LIB_PATH + ".tmp"
    with tempfile.TemporaryDirectory(prefix="cachescout_build_") as work:
        # the control plane: plain host C++ built by the host compiler, with no
        # fused multiply-adds so its fp64 threshold decisions are the
        # expressions as written
        objects = []
        for src in host_sources:
            obj = os.path.join(work, os.path.basename(src) + ".o")
            run([cxx(), "-O2", "-std=c++17", "-fPIC", "-fvisibility=hidden", "-ffp-contract=off",
                 "-Wall", "-Wextra", *includes, "-c", src, "-o", obj], verbose)
            objects.append(obj)
        run([hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
             "-fvisibility=hidden",
             # keep the compiler from forming packed fp32 ops
             "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
             # MFMA accumulators in arch VGPRs: the softmax rescale then works on
             # them in place instead of copying them out of AGPRs every step
             "-mllvm", "-amdgpu-mfma-vgpr-form",
             "-Wall", "-Wno-unused-result", *includes, digest,
             # hipcc compiles every input as HIP unless told otherwise
             *sources, "-x", "none", *objects, "-o", tmp], verbose)
    os.replace(tmp, LIB_PATH)
    return LIB_PATH


if __name__ == "__main__":
    print(build(verbose=True))
