"""The C ABI, on the CPU: the library loads, exports every function the
header declares, and rejects bad arguments before any HIP call.

Only argument combinations that fail validation (or are zero-size no-ops
without events) are passed here; fake device pointers are never dereferenced
because validation returns first.  Nothing here launches a kernel.
"""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "zpp.h")
LIB = os.path.join(ROOT, "paper_2407_01614_amd", "libzpp.so")


@pytest.fixture(scope="module")
def zpp():
    if not os.path.exists(LIB):
        from paper_2407_01614_amd import build
        build.build()
    from paper_2407_01614_amd import zpp as mod
    return mod


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"ZPP_API\s+[\w\s\*]*?\b(zpp_\w+)\s*\(", text)))


def test_header_declares_every_entry_point():
    names = declared_functions()
    for fn in ("zpp_adam_partition_step", "zpp_adam_step_refresh_quantize",
               "zpp_refresh_secondary", "zpp_quantize_blockwise_i8", "zpp_refresh_quantize_i8",
               "zpp_dequant_gather_layer",
               "zpp_quantize_blockwise_i4", "zpp_dequant_reduce_i4", "zpp_qgz_receive_adam_step",
               "zpp_qgz_receive_step_refresh_quantize", "zpp_quantize_blockwise_i4_interleaved",
               "zpp_dequant_reduce_i4_interleaved", "zpp_qgz_receive_adam_step_interleaved",
               "zpp_qgz_receive_step_refresh_quantize_interleaved", "zpp_status_string",
               "zpp_last_hip_error"):
        assert fn in names


def test_library_exports_every_declared_symbol(zpp):
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True,
                         check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for fn in declared_functions():
        assert fn in exported, fn
        assert hasattr(zpp.raw, fn)
    # nothing else of the library's own is exported
    own = {s for s in exported if "zpp" in s.lower()}
    assert own == set(declared_functions())


def test_header_compiles_as_c():
    src = '#include "zpp.h"\nint main(void){ return (int)sizeof(zpp_adam_hparams) - 32; }\n'
    r = subprocess.run(["gcc", "-x", "c", "-std=c99", "-fsyntax-only", "-Wall", "-Werror",
                        "-D__HIP_PLATFORM_AMD__", "-I", os.path.join(ROOT, "include"),
                        "-I", "/opt/rocm/include", "-"], input=src, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_driver_is_built_and_links():
    """The C test driver (built with the library) resolves libzpp.so,
    liboracle.so and the HIP runtime; the GPU test runs it."""
    drv = os.path.join(ROOT, "tests", "c_abi_driver")
    assert os.path.exists(drv), "tests/c_abi_driver is not built: run __graft_entry__.build()"
    out = subprocess.run(["ldd", drv], capture_output=True, text=True, check=True).stdout
    assert "not found" not in out, out
    for lib in ("libzpp.so", "liboracle.so", "libamdhip64.so"):
        assert lib in out, out


def test_hparams_layout(zpp, tmp_path):
    """The binding's mirror of zpp_adam_hparams has the C compiler's layout:
    the same size and every field at the same offset."""
    fields = [f for f, _ in zpp.AdamHParams._fields_]
    src = ('#include <stddef.h>\n#include <stdio.h>\n#include "zpp.h"\nint main(void){\n'
           '  printf("size %zu\\n", sizeof(zpp_adam_hparams));\n'
           + "".join('  printf("%s %%zu\\n", offsetof(zpp_adam_hparams, %s));\n' % (f, f)
                     for f in fields)
           + '  return 0;\n}\n')
    exe = str(tmp_path / "layout")
    r = subprocess.run(["gcc", "-x", "c", "-std=c99", "-D__HIP_PLATFORM_AMD__",
                        "-I", os.path.join(ROOT, "include"), "-I", "/opt/rocm/include", "-",
                        "-o", exe], input=src, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    got = dict(line.split() for line in subprocess.run(
        [exe], capture_output=True, text=True, check=True).stdout.splitlines())
    assert int(got["size"]) == ctypes.sizeof(zpp.AdamHParams) == 32
    for f in fields:
        assert int(got[f]) == getattr(zpp.AdamHParams, f).offset, f


def test_status_strings(zpp):
    for s in range(5):
        assert zpp.raw.zpp_status_string(s)
    assert zpp.raw.zpp_status_string(99) == b"unknown status"


# fake, never-dereferenced device addresses
A = 0x7F0000000000
B = 0x7F0010000000
C = 0x7F0020000000
D = 0x7F0030000000
E = 0x7F0040000000


def hp(zpp, **kw):
    base = dict(lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1, adamw=1, step=1)
    base.update(kw)
    return zpp.AdamHParams(base["lr"], base["beta1"], base["beta2"], base["eps"],
                           base["weight_decay"], base["adamw"], base["step"])


def adam(zpp, ptrs=(A, B, C, D, E), n=1024, h=None):
    h = h if h is not None else hp(zpp)
    return zpp.raw.zpp_adam_partition_step(*ptrs, n, ctypes.byref(h) if h is not False else None,
                                           None)


def test_adam_validation(zpp):
    assert adam(zpp, h=False) == zpp.ZPP_EINVAL
    assert adam(zpp, n=0) == zpp.ZPP_OK  # no-op, nothing enqueued
    assert adam(zpp, ptrs=(None, B, C, D, E)) == zpp.ZPP_EINVAL
    assert adam(zpp, ptrs=(A, B, C, D, None)) == zpp.ZPP_EINVAL
    assert adam(zpp, ptrs=(A + 2, B, C, D, E)) == zpp.ZPP_EALIGN
    assert adam(zpp, ptrs=(A, B, C, D, E + 1)) == zpp.ZPP_EALIGN
    assert adam(zpp, ptrs=(A, A, C, D, E)) == zpp.ZPP_EOVERLAP
    assert adam(zpp, ptrs=(A, B, C, D, A + 4 * 1023)) == zpp.ZPP_EOVERLAP
    assert adam(zpp, ptrs=(A, B, C, B + 4, E)) == zpp.ZPP_EOVERLAP
    for bad in (dict(step=0), dict(beta1=1.0), dict(beta2=-0.1), dict(eps=-1.0),
                dict(lr=float("nan")), dict(weight_decay=float("inf"))):
        assert adam(zpp, h=hp(zpp, **bad)) == zpp.ZPP_EINVAL, bad
    assert adam(zpp, n=(1 << 64) - 1) == zpp.ZPP_EINVAL


F = 0x7F0050000000
G = 0x7F0060000000
H = 0x7F0070000000


def fused(zpp, ptrs=(A, B, C, D, E, F, G, H), n=1024, block=256, h=None):
    h = h if h is not None else hp(zpp)
    return zpp.raw.zpp_adam_step_refresh_quantize(*ptrs, n, block, ctypes.byref(h), None, None,
                                                  None)


def test_fused_validation(zpp):
    assert fused(zpp, n=0) == zpp.ZPP_OK
    assert fused(zpp, n=0, block=100) == zpp.ZPP_EINVAL
    assert fused(zpp, h=hp(zpp, step=0)) == zpp.ZPP_EINVAL
    for blk in (0, 32, 96, 8192):
        assert fused(zpp, block=blk) == zpp.ZPP_EINVAL
    assert fused(zpp, ptrs=(A, B, C, D, None, F, G, H)) == zpp.ZPP_EINVAL
    assert fused(zpp, ptrs=(A, B, C, D, E, F, None, H)) == zpp.ZPP_EINVAL
    assert fused(zpp, ptrs=(A, B, C, D, E, F, G, None)) == zpp.ZPP_EINVAL
    assert fused(zpp, ptrs=(A, B, C, D, E + 1, F, G, H)) == zpp.ZPP_EALIGN
    assert fused(zpp, ptrs=(A, B, C, D, E, F + 1, G, H)) == zpp.ZPP_EALIGN
    assert fused(zpp, ptrs=(A, B, C, D, E, F, G, H + 2)) == zpp.ZPP_EALIGN
    assert fused(zpp, ptrs=(A, B, C, D, E, E + 100, G, H)) == zpp.ZPP_EOVERLAP
    assert fused(zpp, ptrs=(A, B, C, D, E, F, A + 8, H)) == zpp.ZPP_EOVERLAP
    assert fused(zpp, ptrs=(A, B, C, D, E, F, G, G + 1020)) == zpp.ZPP_EOVERLAP


def test_refresh_validation(zpp):
    r = zpp.raw.zpp_refresh_secondary
    assert r(None, None, 0, None, None, None) == zpp.ZPP_OK
    assert r(None, B, 16, None, None, None) == zpp.ZPP_EINVAL
    assert r(A + 1, B, 16, None, None, None) == zpp.ZPP_EALIGN
    assert r(A, A + 30, 16, None, None, None) == zpp.ZPP_EOVERLAP
    assert r(A, A, 16, None, None, None) == zpp.ZPP_EOVERLAP
    assert r(A, B, (1 << 63), None, None, None) == zpp.ZPP_EINVAL


def test_refresh_quantize_validation(zpp):
    rq = zpp.raw.zpp_refresh_quantize_i8
    assert rq(None, None, 0, 256, None, None, None, None, None) == zpp.ZPP_OK
    for blk in (0, 32, 100, 4160):
        assert rq(D, A, 1024, blk, B, C, None, None, None) == zpp.ZPP_EINVAL, blk
    assert rq(None, A, 1024, 256, B, C, None, None, None) == zpp.ZPP_EINVAL
    assert rq(D, A, 1024, 256, None, C, None, None, None) == zpp.ZPP_EINVAL
    assert rq(D + 1, A, 1024, 256, B, C, None, None, None) == zpp.ZPP_EALIGN
    assert rq(D, A + 1, 1024, 256, B, C, None, None, None) == zpp.ZPP_EALIGN
    assert rq(D, A, 1024, 256, B, C + 2, None, None, None) == zpp.ZPP_EALIGN
    assert rq(A + 2046, A, 1024, 256, B, C, None, None, None) == zpp.ZPP_EOVERLAP
    assert rq(D, A, 1024, 256, D + 2047, C, None, None, None) == zpp.ZPP_EOVERLAP
    assert rq(D, A, 1024, 256, B, B + 1020, None, None, None) == zpp.ZPP_EOVERLAP
    assert rq(D, A, 1024, 256, B, A + 2044, None, None, None) == zpp.ZPP_EOVERLAP


def test_quant_validation(zpp):
    q = zpp.raw.zpp_quantize_blockwise_i8
    for blk in (0, 32, 100, 200, 4160, 8192):  # not a multiple of 64 in [64, 4096]
        assert q(A, 1024, blk, B, C, None, None, None) == zpp.ZPP_EINVAL, blk
    assert q(None, 0, 256, None, None, None, None, None) == zpp.ZPP_OK
    assert q(None, 0, 3, None, None, None, None, None) == zpp.ZPP_EINVAL
    assert q(A, 1024, 256, None, C, None, None, None) == zpp.ZPP_EINVAL
    assert q(A + 1, 1024, 256, B, C, None, None, None) == zpp.ZPP_EALIGN
    assert q(A, 1024, 256, B, C + 2, None, None, None) == zpp.ZPP_EALIGN
    assert q(A, 1024, 256, A + 2046, C, None, None, None) == zpp.ZPP_EOVERLAP
    assert q(A, 1024, 256, B, B + 1020, None, None, None) == zpp.ZPP_EOVERLAP
    assert q(A, 1024, 256, B, A + 2044, None, None, None) == zpp.ZPP_EOVERLAP


def gather(zpp, codes, scales, num=None, s=1024, block=256, N=None, out=E, waits=None, nwait=0):
    P = ctypes.c_void_p
    k = len(codes if codes is not None else scales)
    carr = (P * max(k, 1))(*codes) if codes is not None else None
    sarr = (P * max(k, 1))(*scales) if scales is not None else None
    num = k if num is None else num
    N = num * s if N is None else N
    warr = (P * max(nwait, 1))(*(waits or [])) if waits is not None else None
    return zpp.raw.zpp_dequant_gather_layer(carr, sarr, num, s, block, N, out, None, warr, nwait,
                                            None)


def test_gather_validation(zpp):
    cs = [A, B]
    ss = [C, D]
    assert gather(zpp, cs, ss, num=0) == zpp.ZPP_EINVAL
    assert gather(zpp, cs, ss, num=65) == zpp.ZPP_EINVAL
    assert gather(zpp, cs, ss, block=100) == zpp.ZPP_EINVAL
    assert gather(zpp, cs, ss, s=0) == zpp.ZPP_EINVAL
    assert gather(zpp, cs, ss, N=2 * 1024 + 1) == zpp.ZPP_EINVAL
    assert gather(zpp, None, ss) == zpp.ZPP_EINVAL
    assert gather(zpp, [A, None], ss) == zpp.ZPP_EINVAL
    assert gather(zpp, cs, [C, D + 2]) == zpp.ZPP_EALIGN
    assert gather(zpp, cs, ss, out=E + 1) == zpp.ZPP_EALIGN
    assert gather(zpp, cs, ss, out=None) == zpp.ZPP_EINVAL
    assert gather(zpp, cs, ss, out=B + 100) == zpp.ZPP_EOVERLAP
    assert gather(zpp, cs, ss, out=D - 100) == zpp.ZPP_EOVERLAP
    assert gather(zpp, cs, ss, nwait=1, waits=None) == zpp.ZPP_EINVAL
    assert gather(zpp, cs, ss, nwait=1, waits=[None]) == zpp.ZPP_EINVAL
    assert gather(zpp, cs, ss, nwait=65, waits=[A] * 65) == zpp.ZPP_EINVAL
    # an empty layer is a valid no-op (no events given: no HIP call)
    assert gather(zpp, cs, ss, N=0, out=None) == zpp.ZPP_OK


def test_quant_i4_validation(zpp):
    q = zpp.raw.zpp_quantize_blockwise_i4
    assert q(None, 0, 256, None, None, None, None, None) == zpp.ZPP_OK
    for blk in (0, 2, 100, 8192):
        assert q(A, 1024, blk, B, C, None, None, None) == zpp.ZPP_EINVAL
    assert q(A, 1024, 256, None, C, None, None, None) == zpp.ZPP_EINVAL
    assert q(A + 2, 1024, 256, B, C, None, None, None) == zpp.ZPP_EALIGN
    assert q(A, 1024, 256, B, C + 1, None, None, None) == zpp.ZPP_EALIGN
    assert q(A, 1024, 256, A + 4000, C, None, None, None) == zpp.ZPP_EOVERLAP
    assert q(A, 1024, 256, B, B + 508, None, None, None) == zpp.ZPP_EOVERLAP


def reduce_i4(zpp, codes, scales, n=1024, block=256, scale_out=1.0, out=E, waits=None, nwait=0):
    P = ctypes.c_void_p
    k = len(codes)
    carr = (P * k)(*codes)
    sarr = (P * k)(*scales)
    warr = (P * max(nwait, 1))(*(waits or [])) if waits is not None else None
    return zpp.raw.zpp_dequant_reduce_i4(carr, sarr, k, n, block, scale_out, out, None, warr,
                                         nwait, None)


def test_dequant_reduce_i4_validation(zpp):
    cs, ss = [A, B], [C, D]
    assert reduce_i4(zpp, cs, ss, n=0, out=None) == zpp.ZPP_OK
    assert reduce_i4(zpp, cs, ss, block=96) == zpp.ZPP_EINVAL
    assert reduce_i4(zpp, cs, ss, scale_out=float("inf")) == zpp.ZPP_EINVAL
    assert reduce_i4(zpp, [A, None], ss) == zpp.ZPP_EINVAL
    assert reduce_i4(zpp, cs, [C, D + 1]) == zpp.ZPP_EALIGN
    assert reduce_i4(zpp, cs, ss, out=E + 2) == zpp.ZPP_EALIGN
    assert reduce_i4(zpp, cs, ss, out=None) == zpp.ZPP_EINVAL
    assert reduce_i4(zpp, cs, ss, out=A - 100) == zpp.ZPP_EOVERLAP
    assert reduce_i4(zpp, cs, ss, out=D + 8) == zpp.ZPP_EOVERLAP
    assert reduce_i4(zpp, cs, ss, nwait=2, waits=[A, None]) == zpp.ZPP_EINVAL
    assert reduce_i4(zpp, [A] * 65, [C] * 65) == zpp.ZPP_EINVAL


def receive(zpp, state=(A, B, C, E), codes=(F, G), scales=(H, H + 0x1000), n=1024, block=256,
            scale_out=0.5, h=None, waits=None, nwait=0, num=None):
    P = ctypes.c_void_p
    k = len(codes) if num is None else num
    carr = (P * len(codes))(*codes)
    sarr = (P * len(scales))(*scales)
    warr = (P * max(nwait, 1))(*(waits or [])) if waits is not None else None
    h = h if h is not None else hp(zpp)
    return zpp.raw.zpp_qgz_receive_adam_step(state[0], state[1], state[2], carr, sarr, k, block,
                                             scale_out, state[3], n,
                                             ctypes.byref(h) if h is not False else None, None,
                                             warr, nwait, None)


def test_qgz_receive_adam_validation(zpp):
    assert receive(zpp, n=0, state=(None, None, None, None)) == zpp.ZPP_OK
    assert receive(zpp, h=False) == zpp.ZPP_EINVAL
    assert receive(zpp, h=hp(zpp, step=0)) == zpp.ZPP_EINVAL
    assert receive(zpp, h=hp(zpp, beta2=1.0)) == zpp.ZPP_EINVAL
    assert receive(zpp, block=96) == zpp.ZPP_EINVAL
    assert receive(zpp, block=8192) == zpp.ZPP_EINVAL
    assert receive(zpp, scale_out=float("nan")) == zpp.ZPP_EINVAL
    assert receive(zpp, num=0) == zpp.ZPP_EINVAL
    assert receive(zpp, codes=[F] * 65, scales=[H] * 65) == zpp.ZPP_EINVAL
    assert receive(zpp, codes=(F, None)) == zpp.ZPP_EINVAL
    assert receive(zpp, scales=(H, H + 2)) == zpp.ZPP_EALIGN
    assert receive(zpp, state=(A, None, C, E)) == zpp.ZPP_EINVAL
    assert receive(zpp, state=(A + 2, B, C, E)) == zpp.ZPP_EALIGN
    assert receive(zpp, state=(A, B, C, E + 1)) == zpp.ZPP_EALIGN
    assert receive(zpp, state=(A, B, C, A + 64)) == zpp.ZPP_EOVERLAP   # primary in master
    assert receive(zpp, state=(A, A + 4092, C, E)) == zpp.ZPP_EOVERLAP  # moments in master
    assert receive(zpp, codes=(F, A + 16)) == zpp.ZPP_EOVERLAP         # a source in master
    assert receive(zpp, scales=(H, E + 8)) == zpp.ZPP_EOVERLAP         # a scale in primary
    assert receive(zpp, nwait=1, waits=None) == zpp.ZPP_EINVAL
    assert receive(zpp, nwait=2, waits=[A, None]) == zpp.ZPP_EINVAL
    assert receive(zpp, nwait=65, waits=[A] * 65) == zpp.ZPP_EINVAL


def receive_pass(zpp, state=(A, B, C, E, F, G, H), codes=(D, D + 0x100000),
                 scales=(D + 0x200000, D + 0x300000), n=1024, grad_block=256, block=256,
                 scale_out=0.5, h=None, waits=None, nwait=0):
    """state: master, exp_avg, exp_avg_sq, primary, secondary, codes, scales."""
    P = ctypes.c_void_p
    carr = (P * len(codes))(*codes)
    sarr = (P * len(scales))(*scales)
    warr = (P * max(nwait, 1))(*(waits or [])) if waits is not None else None
    h = h if h is not None else hp(zpp)
    return zpp.raw.zpp_qgz_receive_step_refresh_quantize(
        state[0], state[1], state[2], carr, sarr, len(codes), grad_block, scale_out, state[3],
        state[4], state[5], state[6], n, block, ctypes.byref(h) if h is not False else None, None,
        warr, nwait, None)


def test_qgz_receive_pass_validation(zpp):
    assert receive_pass(zpp, n=0, state=(None,) * 7) == zpp.ZPP_OK
    assert receive_pass(zpp, h=False) == zpp.ZPP_EINVAL
    assert receive_pass(zpp, grad_block=96) == zpp.ZPP_EINVAL
    assert receive_pass(zpp, block=32) == zpp.ZPP_EINVAL
    assert receive_pass(zpp, scale_out=float("inf")) == zpp.ZPP_EINVAL
    assert receive_pass(zpp, codes=[D] * 65, scales=[D] * 65) == zpp.ZPP_EINVAL
    assert receive_pass(zpp, codes=(D, None)) == zpp.ZPP_EINVAL
    assert receive_pass(zpp, state=(A, B, C, E, F, None, H)) == zpp.ZPP_EINVAL
    assert receive_pass(zpp, state=(A, B, C, E, F, G, H + 2)) == zpp.ZPP_EALIGN
    assert receive_pass(zpp, state=(A, B, C, E, F + 1, G, H)) == zpp.ZPP_EALIGN
    assert receive_pass(zpp, state=(A, B, C, E, E + 64, G, H)) == zpp.ZPP_EOVERLAP  # sec in prim
    assert receive_pass(zpp, state=(A, B, C, E, F, G, G + 512)) == zpp.ZPP_EOVERLAP  # scales
    assert receive_pass(zpp, codes=(D, A + 16)) == zpp.ZPP_EOVERLAP
    assert receive_pass(zpp, scales=(D + 0x200000, F + 8)) == zpp.ZPP_EOVERLAP
    assert receive_pass(zpp, nwait=1, waits=None) == zpp.ZPP_EINVAL


def quant_il(zpp, src=A, codes=F, scales=H, n=1000, block=256, source=3, num=8):
    return zpp.raw.zpp_quantize_blockwise_i4_interleaved(src, n, block, source, num, codes, scales,
                                                         None, None, None)


def test_quantize_i4_interleaved_validation(zpp):
    """Every case fails validation (or is a size-0 no-op): none reaches a launch."""
    assert quant_il(zpp, n=0, src=None, codes=None, scales=None) == zpp.ZPP_OK
    assert quant_il(zpp, num=0) == zpp.ZPP_EINVAL
    assert quant_il(zpp, num=65) == zpp.ZPP_EINVAL
    assert quant_il(zpp, source=8) == zpp.ZPP_EINVAL
    assert quant_il(zpp, block=100) == zpp.ZPP_EINVAL
    assert quant_il(zpp, n=(1 << 64) // 16 // 8 + 1) == zpp.ZPP_EINVAL
    assert quant_il(zpp, src=None) == zpp.ZPP_EINVAL
    assert quant_il(zpp, src=A + 2) == zpp.ZPP_EALIGN
    assert quant_il(zpp, scales=H + 2) == zpp.ZPP_EALIGN
    assert quant_il(zpp, codes=A + 16) == zpp.ZPP_EOVERLAP        # codes inside src
    assert quant_il(zpp, scales=F + 4000) == zpp.ZPP_EOVERLAP    # scales inside the codes buffer


def reduce_il(zpp, codes=F, scales=H, num=8, n=1024, block=256, scale_out=0.5, out=A,
              waits=None, nwait=0):
    P = ctypes.c_void_p
    warr = (P * max(nwait, 1))(*(waits or [])) if waits is not None else None
    return zpp.raw.zpp_dequant_reduce_i4_interleaved(codes, scales, num, n, block, scale_out, out,
                                                     None, warr, nwait, None)


def test_dequant_reduce_i4_interleaved_validation(zpp):
    """Every case fails validation (or is a size-0 no-op): none reaches a launch."""
    assert reduce_il(zpp, n=0, out=None) == zpp.ZPP_OK
    assert reduce_il(zpp, num=0) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, num=65) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, block=96) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, scale_out=float("nan")) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, n=(1 << 64) // 16 // 8 + 1) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, codes=None) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, scales=None) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, out=None) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, scales=H + 2) == zpp.ZPP_EALIGN
    assert reduce_il(zpp, out=A + 2) == zpp.ZPP_EALIGN
    assert reduce_il(zpp, out=F + 1024) == zpp.ZPP_EOVERLAP      # out inside the codes
    assert reduce_il(zpp, out=H - 16) == zpp.ZPP_EOVERLAP        # out runs into the scales
    assert reduce_il(zpp, nwait=1, waits=None) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, nwait=2, waits=[A, None]) == zpp.ZPP_EINVAL
    assert reduce_il(zpp, nwait=65, waits=[A] * 65) == zpp.ZPP_EINVAL


def receive_il(zpp, state=(A, B, C, E), codes=F, scales=H, num=8, n=1024, block=256,
               scale_out=0.5, h=None, waits=None, nwait=0):
    P = ctypes.c_void_p
    warr = (P * max(nwait, 1))(*(waits or [])) if waits is not None else None
    h = h if h is not None else hp(zpp)
    return zpp.raw.zpp_qgz_receive_adam_step_interleaved(
        state[0], state[1], state[2], codes, scales, num, block, scale_out, state[3], n,
        ctypes.byref(h) if h is not False else None, None, warr, nwait, None)


def test_qgz_receive_interleaved_validation(zpp):
    """Every case fails validation (or is a size-0 no-op): none reaches a launch."""
    assert receive_il(zpp, n=0, state=(None,) * 4) == zpp.ZPP_OK
    assert receive_il(zpp, h=False) == zpp.ZPP_EINVAL
    assert receive_il(zpp, h=hp(zpp, step=0)) == zpp.ZPP_EINVAL
    assert receive_il(zpp, num=0) == zpp.ZPP_EINVAL
    assert receive_il(zpp, num=65) == zpp.ZPP_EINVAL
    assert receive_il(zpp, block=96) == zpp.ZPP_EINVAL
    assert receive_il(zpp, scale_out=float("nan")) == zpp.ZPP_EINVAL
    assert receive_il(zpp, n=(1 << 64) // 16 // 8 + 1) == zpp.ZPP_EINVAL
    assert receive_il(zpp, codes=None) == zpp.ZPP_EINVAL
    assert receive_il(zpp, scales=H + 2) == zpp.ZPP_EALIGN
    assert receive_il(zpp, state=(A, None, C, E)) == zpp.ZPP_EINVAL
    assert receive_il(zpp, state=(A + 2, B, C, E)) == zpp.ZPP_EALIGN
    assert receive_il(zpp, state=(A, B, C, A + 64)) == zpp.ZPP_EOVERLAP  # primary in master
    assert receive_il(zpp, codes=A + 16) == zpp.ZPP_EOVERLAP            # codes in master
    assert receive_il(zpp, scales=E + 8) == zpp.ZPP_EOVERLAP            # scales in primary
    assert receive_il(zpp, nwait=1, waits=None) == zpp.ZPP_EINVAL
    assert receive_il(zpp, nwait=2, waits=[A, None]) == zpp.ZPP_EINVAL
    assert receive_il(zpp, nwait=65, waits=[A] * 65) == zpp.ZPP_EINVAL


def receive_pass_il(zpp, state=(A, B, C, E, F, G, H), codes=D, scales=D + 0x200000, num=8,
                    n=1024, grad_block=256, block=256, scale_out=0.5, h=None, waits=None,
                    nwait=0):
    """state: master, exp_avg, exp_avg_sq, primary, secondary, codes, scales."""
    P = ctypes.c_void_p
    warr = (P * max(nwait, 1))(*(waits or [])) if waits is not None else None
    h = h if h is not None else hp(zpp)
    return zpp.raw.zpp_qgz_receive_step_refresh_quantize_interleaved(
        state[0], state[1], state[2], codes, scales, num, grad_block, scale_out, state[3],
        state[4], state[5], state[6], n, block, ctypes.byref(h) if h is not False else None, None,
        warr, nwait, None)


def test_qgz_receive_pass_interleaved_validation(zpp):
    """Every case fails validation (or is a size-0 no-op): none reaches a launch."""
    assert receive_pass_il(zpp, n=0, state=(None,) * 7) == zpp.ZPP_OK
    assert receive_pass_il(zpp, h=False) == zpp.ZPP_EINVAL
    assert receive_pass_il(zpp, grad_block=96) == zpp.ZPP_EINVAL
    assert receive_pass_il(zpp, block=32) == zpp.ZPP_EINVAL
    assert receive_pass_il(zpp, num=0) == zpp.ZPP_EINVAL
    assert receive_pass_il(zpp, scale_out=float("inf")) == zpp.ZPP_EINVAL
    assert receive_pass_il(zpp, codes=None) == zpp.ZPP_EINVAL
    assert receive_pass_il(zpp, scales=D + 2) == zpp.ZPP_EALIGN
    assert receive_pass_il(zpp, state=(A, B, C, E, F, None, H)) == zpp.ZPP_EINVAL
    assert receive_pass_il(zpp, state=(A, B, C, E, F, G, H + 2)) == zpp.ZPP_EALIGN
    assert receive_pass_il(zpp, state=(A, B, C, E, F + 1, G, H)) == zpp.ZPP_EALIGN
    assert receive_pass_il(zpp, state=(A, B, C, E, E + 64, G, H)) == zpp.ZPP_EOVERLAP
    assert receive_pass_il(zpp, codes=A + 16) == zpp.ZPP_EOVERLAP
    assert receive_pass_il(zpp, scales=F + 8) == zpp.ZPP_EOVERLAP
    assert receive_pass_il(zpp, nwait=1, waits=None) == zpp.ZPP_EINVAL


def test_no_oracle_in_product_path():
    """The product package never reaches for the oracle, nor for any CPU
    fallback of the computation."""
    pkg = os.path.join(ROOT, "paper_2407_01614_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(import|from)\s+oracle|liboracle|zpp_oracle|orc_",
                                     text, re.M), f


CEILING_HEADER = os.path.join(ROOT, "include", "zpp_ceiling.h")
CEILING_LIB = os.path.join(ROOT, "paper_2407_01614_amd", "libzpp_ceiling.so")


def test_ceiling_library_exports_and_rejects():
    """The measurement streams (libzpp_ceiling.so): every function its header
    declares is exported, and bad sizes, alignments or overlaps are
    rejected (hipErrorInvalidValue) before anything is enqueued."""
    if not os.path.exists(CEILING_LIB):
        from paper_2407_01614_amd import build
        build.build_ceiling()
    decl = set(re.findall(r"ZPPC_API\s+int\s+(zppc_\w+)\s*\(", open(CEILING_HEADER).read()))
    assert decl == {"zppc_read_stream", "zppc_write_stream", "zppc_copy_stream",
                    "zppc_adam_pattern", "zppc_gather_pattern", "zppc_quant_pattern"}
    out = subprocess.run(["nm", "-D", "--defined-only", CEILING_LIB], capture_output=True,
                         text=True, check=True).stdout
    exported = {line.split()[-1] for line in out.splitlines() if line.strip()}
    assert {s for s in exported if "zpp" in s.lower()} == decl
    lib = ctypes.CDLL(CEILING_LIB)
    for fn in decl:
        getattr(lib, fn).restype = ctypes.c_int
    EINVAL = 1  # hipErrorInvalidValue
    big = ctypes.c_size_t(1 << 30)
    assert lib.zppc_read_stream(None, big, ctypes.c_void_p(A), None) == EINVAL
    assert lib.zppc_read_stream(ctypes.c_void_p(A), big, None, None) == EINVAL
    assert lib.zppc_read_stream(ctypes.c_void_p(A), ctypes.c_size_t(4000), ctypes.c_void_p(B),
                                None) == EINVAL
    assert lib.zppc_write_stream(ctypes.c_void_p(A + 8), big, ctypes.c_uint32(0), None) == EINVAL
    assert lib.zppc_write_stream(ctypes.c_void_p(A), ctypes.c_size_t(0), ctypes.c_uint32(0),
                                 None) == EINVAL
    assert lib.zppc_copy_stream(ctypes.c_void_p(A), ctypes.c_void_p(A + 4096), big, None) == EINVAL
    assert lib.zppc_copy_stream(ctypes.c_void_p(A), None, big, None) == EINVAL
    P = lambda off=0: ctypes.c_void_p(A + off)
    n = ctypes.c_size_t(1 << 20)
    # the access patterns: sizes that are not whole tiles, misaligned or null
    # pointers
    assert lib.zppc_adam_pattern(P(), P(), P(), P(), P(), ctypes.c_size_t(1000), None) == EINVAL
    assert lib.zppc_adam_pattern(P(), P(8), P(), P(), P(), n, None) == EINVAL
    assert lib.zppc_adam_pattern(P(), P(), P(), P(), P(4), n, None) == EINVAL
    assert lib.zppc_adam_pattern(P(), P(), None, P(), P(), n, None) == EINVAL
    assert lib.zppc_gather_pattern(P(), P(), P(), ctypes.c_size_t(256), None) == EINVAL
    assert lib.zppc_gather_pattern(P(4), P(), P(), n, None) == EINVAL
    assert lib.zppc_gather_pattern(P(), P(2), P(), n, None) == EINVAL
    assert lib.zppc_gather_pattern(P(), P(), P(8), n, None) == EINVAL
    assert lib.zppc_quant_pattern(P(), P(), P(), ctypes.c_size_t(2048), None) == EINVAL
    assert lib.zppc_quant_pattern(P(8), P(), P(), n, None) == EINVAL
    assert lib.zppc_quant_pattern(P(), P(4), P(), n, None) == EINVAL
    assert lib.zppc_quant_pattern(P(), P(), None, n, None) == EINVAL
