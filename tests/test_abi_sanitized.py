"""The C ABI's host-side argument checks under AddressSanitizer and
UndefinedBehaviorSanitizer.

``abi.cpp`` is compiled with g++ for the host only (the kernel launchers are
replaced by stubs that abort if reached) into a sanitized shared library, and
``tests/test_abi_host.py`` runs against it in a child Python with the ASan
runtime preloaded.  Any out-of-bounds access, overflow or undefined
behaviour in the checks fails the child run.
"""

import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _runtime(name):
    out = subprocess.run(["g++", f"-print-file-name={name}"], capture_output=True, text=True)
    path = out.stdout.strip()
    return path if os.path.isabs(path) and os.path.exists(path) else None


@pytest.fixture(scope="module")
def sanitized_lib(tmp_path_factory):
    if shutil.which("g++") is None or _runtime("libasan.so") is None:
        pytest.skip("g++ with the ASan runtime is needed")
    out = str(tmp_path_factory.mktemp("asan") / "libtmamba_host_asan.so")
    cmd = ["g++", "-std=c++17", "-shared", "-fPIC", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           os.path.join(ROOT, "paper_2606_18114_amd", "csrc", "abi.cpp"),
           os.path.join(ROOT, "tests", "abi_launch_stubs.cpp"),
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", "-o", out]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    assert proc.returncode == 0, proc.stderr
    return out


def test_abi_checks_under_sanitizers(sanitized_lib):
    env = dict(os.environ)
    env["LD_PRELOAD"] = _runtime("libasan.so")
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=1"
    env["UBSAN_OPTIONS"] = "print_stacktrace=1:halt_on_error=1"
    env["TM_ABI_TEST_LIB"] = sanitized_lib
    proc = subprocess.run([sys.executable, "-m", "pytest", "-q", "-p", "no:cacheprovider",
                           os.path.join(ROOT, "tests", "test_abi_host.py")],
                          capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    assert proc.returncode == 0, proc.stdout[-3000:] + proc.stderr[-3000:]
    assert "passed" in proc.stdout
