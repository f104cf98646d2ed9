"""The host code of the C ABI and the control plane under AddressSanitizer
and UndefinedBehaviorSanitizer.

Builds the library with both sanitizers on its host side
(``paper_2608_14624_amd/build_sanitized.py``; device code unchanged) and runs
the host ABI tests and the control-plane tests against that build in a child
process with the sanitizer runtime preloaded.  Any report aborts the child.
"""

import shutil
import subprocess

import pytest

from paper_2608_14624_amd import build_sanitized


@pytest.mark.slow
def test_abi_and_control_plane_tests_pass_under_asan_and_ubsan():
    if shutil.which("hipcc") is None and not shutil.which("/opt/rocm/bin/hipcc"):
        pytest.skip("hipcc not available")
    lib = build_sanitized.build()
    nm = shutil.which("nm")
    if nm is not None:
        syms = subprocess.run([nm, "-D", lib], capture_output=True, text=True, check=True).stdout
        assert "__asan_report_load" in syms and "__ubsan_handle" in syms, "not instrumented"
    assert build_sanitized.run_tests() == 0
