"""The C ABI's host code (abi.cpp) under AddressSanitizer and
UndefinedBehaviorSanitizer, on the CPU: abi.cpp is built for the host with
g++ next to stand-ins for the kernel launchers that record their arguments
(tests/asan/abi_stubs.cpp) and a driver that calls every entry point
(tests/asan/abi_driver.cpp).  No GPU code is built or run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_01651_amd", "csrc")
HERE = os.path.join(ROOT, "tests", "asan")


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_abi_host_code_under_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_driver")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{ROOT}/include", f"-I{CSRC}", f"-I{HERE}",
           os.path.join(CSRC, "abi.cpp"), os.path.join(HERE, "abi_stubs.cpp"),
           os.path.join(HERE, "abi_driver.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, (r.stdout + r.stderr)[-4000:]
    assert "all checks held" in r.stdout
