"""Host-side sanitizer runs (CPU only): the fp64 oracle and the library's
host code (the C ABI: validation, work splitting, workspace layout, error
paths) built with AddressSanitizer and UndefinedBehaviorSanitizer by the
host compilers, with every finding fatal, and driven by the programs under
tests/sanitize/. The host code is linked with launch stand-ins, so no GPU
code is built or run here."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
       "-fno-omit-frame-pointer"]
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


def _run(exe, leaks):
    env = dict(os.environ, ASAN_OPTIONS=f"detect_leaks={1 if leaks else 0}:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1", OMP_NUM_THREADS="2")
    res = subprocess.run([exe], capture_output=True, text=True, timeout=300, env=env)
    assert res.returncode == 0, res.stdout + res.stderr
    assert "ERROR: AddressSanitizer" not in res.stderr and "runtime error" not in res.stderr, res.stderr
    return res.stdout


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc missing")
def test_oracle_under_address_and_undefined_behavior_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_san")
    subprocess.check_call(["gcc", "-std=c11", *SAN, "-fopenmp", "-Wall", "-Werror",
                           os.path.join(ROOT, "oracle", "oracle.c"),
                           os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c"),
                           "-o", exe, "-lm"])
    assert "all checks passed" in _run(exe, leaks=True)


@pytest.mark.skipif(shutil.which("g++") is None or
                    not os.path.exists(os.path.join(ROCM, "lib", "libamdhip64.so")),
                    reason="g++ or the HIP runtime missing")
def test_host_abi_under_address_and_undefined_behavior_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_san")
    csrc = os.path.join(ROOT, "paper_2403_08845_amd", "csrc")
    subprocess.check_call(["g++", "-std=c++17", *SAN, "-Wall", "-D__HIP_PLATFORM_AMD__",
                           f"-I{ROCM}/include", f"-I{ROOT}/include", f"-I{csrc}",
                           os.path.join(csrc, "bifattn_host.cpp"),
                           os.path.join(ROOT, "tests", "sanitize", "launch_stubs.cpp"),
                           os.path.join(ROOT, "tests", "sanitize", "abi_driver.cpp"),
                           f"-L{ROCM}/lib", "-lamdhip64", f"-Wl,-rpath,{ROCM}/lib", "-o", exe])
    # the HIP runtime keeps allocations for the process's lifetime: leaks off
    assert "all checks passed" in _run(exe, leaks=False)
