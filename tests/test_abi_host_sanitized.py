"""The C ABI's host layer (argument checks, workspace sizing, launch planning)
built with AddressSanitizer and UndefinedBehaviorSanitizer and driven through
every entry point: documented error cases, valid calls (which reach stub
launchers; no GPU code is built) and many random argument sets.

The build uses g++ on the host sources only (csrc/lt_api.cpp, csrc/plan.cpp)
plus tests/abi_host_check.cpp; any sanitizer report aborts the program.
"""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_10415_amd", "csrc")
ROCM = "/opt/rocm"


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir(f"{ROCM}/include/hip"),
                    reason="needs g++ and the HIP headers")
def test_abi_host_layer_under_sanitizers(tmp_path):
    exe = tmp_path / "abi_host_check"
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", f"-I{ROCM}/include", f"-I{ROOT}/include",
           os.path.join(CSRC, "lt_api.cpp"), os.path.join(CSRC, "plan.cpp"),
           os.path.join(ROOT, "tests", "abi_host_check.cpp"),
           f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-o", str(exe)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([str(exe), "20000"], capture_output=True, text=True, env=env, timeout=600)
    print(r.stdout)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-6000:])
    assert "0 failures" in r.stdout
