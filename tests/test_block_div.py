"""The block index of the kernels (BlockDiv in csrc/zpp_launch.h) equals
i / block for every block size the library accepts, checked on the host by
tests/block_div_check.cpp (the device's __umul64hi is the high half of the
same 128-bit product)."""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
CLANGXX = os.path.join(ROCM, "llvm", "bin", "clang++")


@pytest.mark.skipif(not os.path.exists(CLANGXX), reason="ROCm clang++ not found")
def test_block_index_is_exact(tmp_path):
    exe = str(tmp_path / "block_div_check")
    cmd = [CLANGXX, "-std=c++17", "-O2", "-D__HIP_PLATFORM_AMD__",
           "-I", os.path.join(ROOT, "paper_2407_01614_amd", "csrc"),
           "-I", os.path.join(ROCM, "include"), os.path.join(HERE, "block_div_check.cpp"),
           "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "block index ok" in r.stdout, r.stdout + r.stderr


@pytest.mark.skipif(not os.path.exists(CLANGXX), reason="ROCm clang++ not found")
def test_work_shapes_cover_every_element(tmp_path):
    """The lane groups of the quantizers for blocks that are not powers of two
    and the per-XCD workgroup renumbering (csrc/zpp_chunk.h), checked on the
    host by tests/work_shape_check.cpp."""
    exe = str(tmp_path / "work_shape_check")
    cmd = [CLANGXX, "-std=c++17", "-O2", "-I", os.path.join(ROOT, "paper_2407_01614_amd", "csrc"),
           os.path.join(HERE, "work_shape_check.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, " ".join(cmd) + "\n" + r.stderr
    r = subprocess.run([exe], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0 and "work shapes ok" in r.stdout, r.stdout + r.stderr
