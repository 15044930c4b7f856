"""The C ABI's host code under AddressSanitizer and UndefinedBehaviorSanitizer
(CPU): csrc/zpp_api.hip (argument checks, event ordering, dispatch) is built
as host C++ with the sanitizers, linked with counting stand-ins for the
kernel launchers, and driven by tests/abi_sanitizer_driver.c through every
entry point's validation paths and size-0 calls, with host-side pointer and
event arrays of exactly the stated lengths.  No case may reach a launcher."""
import glob
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
CLANG = os.path.join(ROCM, "llvm", "bin", "clang")
CLANGXX = os.path.join(ROCM, "llvm", "bin", "clang++")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
       "-fno-omit-frame-pointer", "-O1", "-g"]


def have_toolchain():
    rt = glob.glob(os.path.join(ROCM, "llvm", "lib", "clang", "*", "lib", "linux",
                                "libclang_rt.asan-x86_64.a"))
    return (os.path.exists(CLANG) and os.path.exists(CLANGXX) and bool(rt)
            and os.path.exists(os.path.join(ROCM, "lib", "libamdhip64.so")))


@pytest.mark.skipif(not have_toolchain(), reason="ROCm clang with sanitizer runtimes not found")
def test_abi_host_code_clean_under_sanitizers(tmp_path):
    inc = ["-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
           "-I", os.path.join(ROOT, "paper_2407_01614_amd", "csrc"),
           "-I", os.path.join(ROCM, "include")]
    api, stubs, drv = (str(tmp_path / x) for x in ("api.o", "stubs.o", "driver.o"))
    exe = str(tmp_path / "abi_sanitized")
    steps = [
        [CLANGXX, "-x", "c++", "-std=c++17", *SAN, *inc, "-c",
         os.path.join(ROOT, "paper_2407_01614_amd", "csrc", "zpp_api.hip"), "-o", api],
        [CLANGXX, "-std=c++17", *SAN, *inc, "-c", os.path.join(HERE, "abi_launch_stubs.cpp"),
         "-o", stubs],
        [CLANG, "-std=c11", *SAN, *inc, "-c", os.path.join(HERE, "abi_sanitizer_driver.c"),
         "-o", drv],
        [CLANGXX, *SAN, api, stubs, drv, "-L", os.path.join(ROCM, "lib"), "-lamdhip64",
         "-Wl,-rpath," + os.path.join(ROCM, "lib"), "-o", exe],
    ]
    for cmd in steps:
        r = subprocess.run(cmd, capture_output=True, text=True)
        assert r.returncode == 0, " ".join(cmd) + "\n" + r.stderr
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "sanitized abi run ok" in r.stdout
