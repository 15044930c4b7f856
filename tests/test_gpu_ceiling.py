"""The measurement streams of libzpp_ceiling.so on the GPU: each writes
exactly what its header says over exactly its range (guard words past the
end stay untouched), so the bytes bench.py credits them with are the bytes
they move."""
import ctypes
import os

import numpy as np
import pytest
import torch

from paper_2407_01614_amd.build import CEILING_LIB

pytestmark = pytest.mark.gpu

GUARD = 4096  # bytes of sentinel after every output


@pytest.fixture(scope="module")
def lib():
    assert os.path.exists(CEILING_LIB), "libzpp_ceiling.so is not built"
    L = ctypes.CDLL(CEILING_LIB)
    for fn in ("zppc_read_stream", "zppc_write_stream", "zppc_copy_stream", "zppc_adam_pattern",
               "zppc_gather_pattern", "zppc_quant_pattern"):
        getattr(L, fn).restype = ctypes.c_int
    return L


def vp(t):
    return ctypes.c_void_p(t.data_ptr())


def guarded(nbytes, fill=0xA5):
    """A device byte buffer of nbytes + GUARD, all set to `fill`."""
    return torch.full((nbytes + GUARD,), fill, dtype=torch.uint8, device="cuda")


def rand_bytes(nbytes, seed):
    g = np.random.default_rng(seed)
    return torch.from_numpy(g.integers(0, 256, nbytes, dtype=np.uint8)).cuda()


def host(t):
    torch.cuda.synchronize()
    return t.cpu().numpy()


def assert_guard(buf, nbytes, fill=0xA5):
    assert (host(buf)[nbytes:] == fill).all(), "a stream wrote past its range"


def test_copy_and_write_streams(lib):
    nbytes = 3 * 4096
    src = rand_bytes(nbytes, 1)
    dst = guarded(nbytes)
    assert lib.zppc_copy_stream(vp(dst), vp(src), ctypes.c_size_t(nbytes), None) == 0
    assert (host(dst)[:nbytes] == host(src)).all()
    assert_guard(dst, nbytes)
    dst = guarded(nbytes)
    assert lib.zppc_write_stream(vp(dst), ctypes.c_size_t(nbytes), ctypes.c_uint32(0x3F803F80),
                                 None) == 0
    assert (host(dst)[:nbytes].view(np.uint32) == 0x3F803F80).all()
    assert_guard(dst, nbytes)


def test_read_stream_leaves_sink(lib):
    nbytes = 5 * 4096
    src = torch.ones(nbytes // 2, dtype=torch.int16, device="cuda")
    sink = torch.full((1,), 7, dtype=torch.int32, device="cuda")
    assert lib.zppc_read_stream(vp(src), ctypes.c_size_t(nbytes), vp(sink), None) == 0
    assert int(host(sink)[0]) == 7


def test_adam_pattern(lib):
    n = 256 * 37
    arrays = [rand_bytes(4 * n, 10 + k) for k in range(4)]
    p, m, v, g = (guarded(4 * n) for _ in range(4))
    for buf, a in zip((p, m, v, g), arrays):
        buf[:4 * n].copy_(a)
    out = guarded(2 * n)
    assert lib.zppc_adam_pattern(vp(p), vp(m), vp(v), vp(g), vp(out), ctypes.c_size_t(n),
                                 None) == 0
    P, M, V, G = (host(a).view(np.uint32) for a in arrays)
    assert (host(p)[:4 * n].view(np.uint32) == (P ^ G)).all()
    assert (host(m)[:4 * n].view(np.uint32) == (M ^ G)).all()
    assert (host(v)[:4 * n].view(np.uint32) == (V ^ G)).all()
    assert (host(g)[:4 * n] == host(arrays[3])).all()
    P1 = (P ^ G).reshape(-1, 2)
    words = (P1[:, 0] >> 16) | (P1[:, 1] & 0xFFFF0000)
    assert (host(out)[:2 * n].view(np.uint32) == words).all()
    for buf, nb in ((p, 4 * n), (m, 4 * n), (v, 4 * n), (g, 4 * n), (out, 2 * n)):
        assert_guard(buf, nb)


def test_gather_pattern(lib):
    n = 512 * 29
    codes = rand_bytes(n, 20)
    scales = rand_bytes(4 * (n // 256), 21)
    out = guarded(2 * n)
    assert lib.zppc_gather_pattern(vp(codes), vp(scales), vp(out), ctypes.c_size_t(n),
                                   None) == 0
    c = host(codes).view(np.uint32).reshape(n // 512, 64, 2)     # row, lane, word
    s = host(scales).view(np.uint32).reshape(n // 512, 2)        # the row's two scales
    lane_s = np.where(np.arange(64)[None, :] < 32, s[:, :1], s[:, 1:])
    want = np.stack([c[..., 0], c[..., 1], c[..., 0] ^ lane_s, c[..., 1] ^ lane_s], axis=-1)
    assert (host(out)[:2 * n].view(np.uint32).reshape(want.shape) == want).all()
    assert_guard(out, 2 * n)


def test_quant_pattern(lib):
    n = 4096 * 7
    src = rand_bytes(2 * n, 30)
    codes = guarded(n)
    scales = guarded(4 * (n // 256))
    assert lib.zppc_quant_pattern(vp(src), vp(codes), vp(scales), ctypes.c_size_t(n), None) == 0
    x = host(src).view(np.uint32).reshape(n // 256, 32, 4)     # block, lane, word
    want = np.stack([x[..., 0] ^ x[..., 2], x[..., 1] ^ x[..., 3]], axis=-1)
    assert (host(codes)[:n].view(np.uint32).reshape(want.shape) == want).all()
    assert (host(scales)[:4 * (n // 256)].view(np.uint32) == (x[:, 0, 0] & 0x3FFFFFFF)).all()
    assert_guard(codes, n)
    assert_guard(scales, 4 * (n // 256))
