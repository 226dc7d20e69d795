"""The library's host code under AddressSanitizer and UndefinedBehaviorSanitizer.

The C ABI's host side (argument checks, the host plan of a batch, the host
adapter packer, the sizing functions) is compiled with g++ and both
sanitizers, the kernel launchers replaced by stubs, and driven on random
inputs by tests/host_sanitize/driver.cpp, which also checks every result
against a plain re-statement.  Any invalid access, leak-free-use error or
undefined behaviour aborts the run.  CPU only (no GPU, no device code)."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir(os.path.join(ROCM, "include", "hip")),
                    reason="needs g++ and the HIP headers")
def test_host_code_is_clean_under_asan_and_ubsan(tmp_path):
    exe = str(tmp_path / "host_sanitize")
    src = [os.path.join(ROOT, "tests", "host_sanitize", "driver.cpp"),
           os.path.join(ROOT, "tests", "host_sanitize", "launch_stubs.cpp"),
           os.path.join(ROOT, "paper_2510_23346_amd", "csrc", "bdl_api.cpp")]
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROCM, "include"), "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2510_23346_amd", "csrc")] + src + [
           "-L", os.path.join(ROCM, "lib"), "-lamdhip64", f"-Wl,-rpath,{os.path.join(ROCM, 'lib')}", "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    # the sanitizer runtimes are really in the binary
    nm = subprocess.run(["nm", exe], capture_output=True, text=True).stdout
    assert "__asan_init" in nm and "__ubsan_handle" in nm
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=0", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "0 failed checks" in r.stdout
