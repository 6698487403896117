"""Host code of the library (assignment, row tables, clique enumeration, the
multithreaded simulator, argument checks) and the oracle built with g++
under AddressSanitizer and UndefinedBehaviorSanitizer, with the device
launchers stubbed out, and run on the CPU (tests/host_sanitize/)."""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "host_sanitize")
ROOT = os.path.dirname(HERE)
ROCM = "/opt/rocm"


@pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None
                    or not os.path.exists(os.path.join(ROCM, "lib", "libamdhip64.so")),
                    reason="needs gcc/g++ and the ROCm host runtime library")
def test_host_code_under_sanitizers(tmp_path):
    san = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-fno-omit-frame-pointer", "-g", "-O1"]
    obj = tmp_path / "oracle.o"
    subprocess.run(["gcc", "-std=c11", *san, "-c", os.path.join(ROOT, "oracle", "oracle.c"),
                    "-o", str(obj)], check=True)
    exe = tmp_path / "host_sanitize"
    srcs = [os.path.join(SRC, "driver.cpp"), os.path.join(SRC, "device_stubs.cpp"),
            os.path.join(ROOT, "paper_2108_02416_amd", "csrc", "aspis_host.cpp"),
            os.path.join(ROOT, "paper_2108_02416_amd", "csrc", "aspis_sim.cpp")]
    subprocess.run(["g++", "-std=c++17", *san, "-D__HIP_PLATFORM_AMD__",
                    "-I", os.path.join(ROCM, "include"), *srcs, str(obj),
                    "-L", os.path.join(ROCM, "lib"), f"-Wl,-rpath,{ROCM}/lib", "-lamdhip64",
                    "-lpthread", "-o", str(exe)], check=True)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    out = subprocess.run([str(exe)], capture_output=True, text=True, env=env, timeout=300)
    assert out.returncode == 0, out.stdout + out.stderr
    assert out.stdout.strip().endswith("ok")
    assert "runtime error" not in out.stderr and "AddressSanitizer" not in out.stderr, out.stderr
