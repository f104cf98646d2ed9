"""Build libcachescout.so with AddressSanitizer and UndefinedBehaviorSanitizer
on its host code, for the CPU tests of the C ABI and the control plane.

    python -m paper_2608_14624_amd.build_sanitized [--run-tests]

The device code is built as usual (sanitizers apply to the host side only:
each ``-fsanitize=`` follows ``-Xarch_host`` on the hipcc line; the
host-only control plane is built by clang++ with the same sanitizers).  The
library goes to ``_build/sanitized/libcachescout.so``; the in-tree library is
left alone.  To use it, preload the sanitizer runtime into the Python process
and point the binding at the sanitized build:

    LD_PRELOAD=<libclang_rt.asan> ASAN_OPTIONS=detect_leaks=0 \\
    CACHESCOUT_LIB=_build/sanitized/libcachescout.so python -m pytest ...

``--run-tests`` does that for the host ABI and control-plane test files.
"""

import os
import subprocess
import sys
import tempfile

from . import build as _build

OUT_DIR = os.path.join(_build.ROOT, "_build", "sanitized")
OUT_LIB = os.path.join(OUT_DIR, _build.LIB_NAME)
SANITIZE = "-fsanitize=address,undefined"
TESTS = ("tests/test_abi_host.py", "tests/test_control_plane.py")


def clangxx():
    path = os.path.join(os.path.dirname(os.path.realpath(_build.hipcc())), "..", "llvm", "bin",
                        "clang++")
    for cand in (path, "/opt/rocm/llvm/bin/clang++"):
        if os.path.exists(cand):
            return os.path.realpath(cand)
    raise RuntimeError("clang++ of the ROCm toolchain not found")


def asan_runtime():
    out = subprocess.run([clangxx(), "-print-file-name=libclang_rt.asan-x86_64.so"],
                         capture_output=True, text=True, check=True).stdout.strip()
    if not os.path.exists(out):
        raise RuntimeError(f"ASan runtime not found ({out})")
    return out


def build(verbose=False):
    sources = sorted(f for f in _build.source_files() if f.endswith(".hip"))
    host_sources = sorted(f for f in _build.source_files() if f.endswith(".cpp"))
    includes = ["-I", os.path.join(_build.ROOT, "include"), "-I", os.path.join(_build.PKG_DIR, "csrc")]
    digest = f'-DCS_SOURCE_DIGEST="{_build.source_digest()}"'
    os.makedirs(OUT_DIR, exist_ok=True)
    with tempfile.TemporaryDirectory(prefix="cachescout_asan_") as work:
        objects = []
        for src in host_sources:
            obj = os.path.join(work, os.path.basename(src) + ".o")
            _build.run([clangxx(), "-O1", "-g", "-std=c++17", "-fPIC", "-fvisibility=hidden",
                        "-ffp-contract=off", "-fno-omit-frame-pointer", SANITIZE,
                        "-fno-sanitize-recover=all", *includes, "-c", src, "-o", obj], verbose)
            objects.append(obj)
        _build.run([_build.hipcc(), f"--offload-arch={_build.ARCH}", "-O1", "-g", "-std=c++17",
                    "-fPIC", "-shared", "-fvisibility=hidden",
                    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                    "-mllvm", "-amdgpu-mfma-vgpr-form",
                    "-Xarch_host", SANITIZE, "-Xarch_host", "-fno-sanitize-recover=all",
                    "-Xarch_host", "-fno-omit-frame-pointer",
                    "-Wall", "-Wno-unused-result", *includes, digest,
                    *sources, "-x", "none", *objects, "-o", OUT_LIB], verbose)
    return OUT_LIB


def run_tests(extra=()):
    env = dict(os.environ)
    env["LD_PRELOAD"] = asan_runtime()
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["CACHESCOUT_LIB"] = OUT_LIB
    cmd = [sys.executable, "-m", "pytest", "-q", "-m", "not gpu", "-p", "no:cacheprovider",
           *TESTS, *extra]
    return subprocess.run(cmd, cwd=_build.ROOT, env=env).returncode


if __name__ == "__main__":
    print(build(verbose=True), flush=True)
    if "--run-tests" in sys.argv:
        sys.exit(run_tests())
