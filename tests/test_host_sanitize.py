"""The C ABI's host layer under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU only).  capi.hip is rebuilt with both sanitizers on its host code (its
device code and every other object unchanged) and linked into a native driver,
tests/sanitize/abi_host_checks.cpp, that runs the host-only calls (budget
assignment, the Eq. 2 policy, budget split, workspace sizes) over their whole
range and every device call's argument validation, which returns before any
HIP call.  A sanitizer finding aborts the driver."""
import glob
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_29029_amd")
CLANG = "/opt/rocm/llvm/bin/clang++"

pytestmark = pytest.mark.slow


def _tools():
    from paper_2609_29029_amd.build import hipcc
    if not os.path.exists(CLANG):
        pytest.skip("no ROCm clang++ in this image")
    return hipcc()


def test_host_layer_under_asan_and_ubsan(tmp_path):
    hipcc = _tools()
    from paper_2609_29029_amd import build as B
    if not all(os.path.exists(os.path.join(B.BUILD, s.replace(".hip", ".o"))) for s in B.SOURCES):
        B.build()
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    capi_o = str(tmp_path / "capi_san.o")
    r = subprocess.run([hipcc, "-O1", "-g", "-std=c++17", f"--offload-arch={B.ARCH}", "-fPIC", *san,
                        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                        "-c", os.path.join(B.CSRC, "capi.hip"), "-o", capi_o], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    drv_o = str(tmp_path / "driver.o")
    host_san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer"]
    r = subprocess.run([CLANG, "-O1", "-g", "-std=c++17", *host_san, "-c",
                        os.path.join(ROOT, "tests", "sanitize", "abi_host_checks.cpp"), "-o", drv_o],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    others = [os.path.join(B.BUILD, s.replace(".hip", ".o")) for s in B.SOURCES if s != "capi.hip"]
    exe = str(tmp_path / "abi_host_checks")
    r = subprocess.run([CLANG, *host_san, drv_o, capi_o, *others, "-L/opt/rocm/lib", "-lamdhip64",
                        "-Wl,-rpath,/opt/rocm/lib", "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    env = dict(os.environ, ASAN_OPTIONS="abort_on_error=1:detect_leaks=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    print(r.stdout, r.stderr[-4000:])
    assert r.returncode == 0, r.stderr[-4000:]
    assert " 0 failed" in r.stdout
