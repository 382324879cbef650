"""The C ABI's error paths with the host runtime under AddressSanitizer: the
runtime's *.cpp files are rebuilt with the sanitizer (kernels unchanged),
tests/abi_checks.c drives NULL contexts, rejected initialisations and a
context whose initialisation failed, and any invalid host memory access
aborts the program.  Runs without a GPU."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang"


def test_abi_error_paths_under_address_sanitizer(tmp_path):
    if not (os.path.exists(CLANG) or shutil.which("clang")):
        pytest.skip("no clang for the sanitizer build")
    from paper_1903_12287_amd import build
    lib = build.build_asan()
    exe = str(tmp_path / "abi_checks")
    libdir = os.path.dirname(lib)
    cc = CLANG if os.path.exists(CLANG) else shutil.which("clang")
    r = subprocess.run([cc, "-fsanitize=address", "-fno-omit-frame-pointer", "-g", "-I", os.path.join(ROOT, "include"),
                        os.path.join(ROOT, "tests", "abi_checks.c"), "-o", exe, f"-L{libdir}", "-lpbg_asan",
                        f"-Wl,-rpath,{libdir}"], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ)
    # the HIP runtime keeps allocations until exit; only access errors count
    env["ASAN_OPTIONS"] = "detect_leaks=0:abort_on_error=0:halt_on_error=1"
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "abi checks passed" in r.stdout
    assert "AddressSanitizer" not in r.stderr
