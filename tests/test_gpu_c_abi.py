"""The C ABI used from plain C: tests/c_abi_driver (built with the library by
the repository's build step) runs one iteration of the path with hipMalloc'd
buffers, three streams and caller-owned events, and checks it against the
oracle's C library; then the qgZ receive fused into the partition step,
against the dequantize-and-reduce followed by the step, from separate int4
arrays and from one interleaved receive buffer.  It runs as a child process
of the test runner."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu

DRIVER = os.path.join(os.path.dirname(os.path.abspath(__file__)), "c_abi_driver")


@pytest.mark.parametrize("n", [(1 << 20) + 4096, 300 * 256 + 40])
def test_c_driver(n):
    assert os.path.exists(DRIVER), "tests/c_abi_driver is not built: run __graft_entry__.build()"
    print("c driver n=%d" % n, flush=True)
    r = subprocess.run([DRIVER, str(n)], capture_output=True, text=True, timeout=100)
    sys.stdout.write(r.stdout)
    sys.stderr.write(r.stderr)
    assert r.returncode == 0, r.stderr[-2000:]
    assert "c abi ok" in r.stdout
