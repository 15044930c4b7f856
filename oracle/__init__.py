"""CPU oracle for the one-rank partition path of modified ZeRO++ hpZ
(arXiv 2407.01614).

TEST INFRASTRUCTURE ONLY: the test suite, the smoke check and the benchmark's
CPU-baseline leg may import this package; the product path never does.  The
arithmetic lives in ``zpp_oracle.c`` (scalar C, binary64 for the optimizer,
binary32 where a float decides an integer code).  This module only marshals
numpy arrays into it and holds the partition-size rule of Eq. 1.

Every function here is pinned by ``tests/test_oracle_pins.py`` against
something other than itself (library routines, closed forms, exact integer
constructions, brute force, invariants).
"""
import ctypes
import os

import numpy as np

from . import build as _build


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p)


def _req(a, dtype):
    a = np.asarray(a)
    if a.dtype != dtype:
        raise TypeError("expected %s, got %s" % (dtype, a.dtype))
    return np.ascontiguousarray(a)


def num_blocks(n, block):
    return (n + block - 1) // block


class Oracle:
    """numpy front end over one build of ``zpp_oracle.c``."""

    def __init__(self, lib_path):
        lib = ctypes.CDLL(lib_path)
        P = ctypes.c_void_p
        sz = ctypes.c_size_t
        u32 = ctypes.c_uint32
        f32 = ctypes.c_float
        lib.orc_bf16_rne.restype = ctypes.c_uint16
        lib.orc_bf16_rne.argtypes = [f32]
        lib.orc_bf16_rne_array.argtypes = [P, P, sz]
        lib.orc_bf16_to_f32_array.argtypes = [P, P, sz]
        lib.orc_adam_step.argtypes = [P, P, P, P, P, sz, f32, f32, f32, f32, f32,
                                      ctypes.c_int64, ctypes.c_int]
        lib.orc_refresh.argtypes = [P, P, sz]
        lib.orc_quantize_blockwise_i8.argtypes = [P, sz, u32, P, P]
        lib.orc_dequant_blockwise_i8.argtypes = [P, P, sz, u32, P]
        lib.orc_dequant_gather_layer.argtypes = [P, P, u32, sz, u32, sz, P]
        lib.orc_quantize_blockwise_i4.argtypes = [P, sz, u32, P, P]
        lib.orc_unpack_i4.argtypes = [P, sz, P]
        lib.orc_dequant_reduce_i4.argtypes = [P, P, u32, sz, u32, f32, P]
        self.lib = lib
        self.path = lib_path

    # -- bf16 conversions ---------------------------------------------------
    def bf16_rne(self, x):
        """float32 array -> uint16 bf16 bits, round-to-nearest-even, NaN -> 0x7FC0."""
        x = _req(x, np.float32)
        out = np.empty(x.shape, np.uint16)
        self.lib.orc_bf16_rne_array(_ptr(x), _ptr(out), x.size)
        return out

    def bf16_to_f32(self, h):
        """uint16 bf16 bits -> float32 (exact)."""
        h = _req(h, np.uint16)
        out = np.empty(h.shape, np.float32)
        self.lib.orc_bf16_to_f32_array(_ptr(h), _ptr(out), h.size)
        return out

    # -- partition step (Algorithm 1: optimizer.step on the rank's partition)
    def adam_step(self, p, m, v, g, lr, beta1, beta2, eps, weight_decay, step, adamw=True,
                  emit=True):
        """One Adam(W) step.  Returns new (p, m, v, bf16_bits) as fresh arrays;
        the inputs are left alone.  ``step`` is Adam's 1-based t."""
        p = _req(p, np.float32).copy()
        m = _req(m, np.float32).copy()
        v = _req(v, np.float32).copy()
        g = _req(g, np.float32)
        n = p.size
        if not (m.size == v.size == g.size == n):
            raise ValueError("p, m, v, g sizes differ")
        if step < 1:
            raise ValueError("step is 1-based")
        out = np.empty(n, np.uint16) if emit else None
        self.lib.orc_adam_step(_ptr(p), _ptr(m), _ptr(v), _ptr(g),
                               _ptr(out) if emit else None, n, lr, beta1, beta2, eps,
                               weight_decay, int(step), 1 if adamw else 0)
        return p, m, v, out

    # -- secondary refresh (Algorithm 1 forward loop; Eq. 1) ------------------
    def refresh(self, src):
        src = _req(src, np.uint16)
        dst = np.empty_like(src)
        self.lib.orc_refresh(_ptr(dst), _ptr(src), src.size)
        return dst

    # -- qwZ blockwise int8 quantization and its inverse ---------------------
    def quantize_blockwise_i8(self, x_bf16, block=256):
        x = _req(x_bf16, np.uint16)
        codes = np.empty(x.size, np.int8)
        scales = np.empty(num_blocks(x.size, block), np.float32)
        self.lib.orc_quantize_blockwise_i8(_ptr(x), x.size, block, _ptr(codes), _ptr(scales))
        return codes, scales

    def dequant_blockwise_i8(self, codes, scales, block=256):
        codes = _req(codes, np.int8)
        scales = _req(scales, np.float32)
        if scales.size < num_blocks(codes.size, block):
            raise ValueError("too few scales")
        out = np.empty(codes.size, np.uint16)
        self.lib.orc_dequant_blockwise_i8(_ptr(codes), _ptr(scales), codes.size, block,
                                          _ptr(out))
        return out

    def dequant_gather_layer(self, shard_codes, shard_scales, shard_elems, block, layer_elems):
        """Backward AllGather(L, P') with dequantization: the in-order
        concatenation of the dequantized shards, cut at ``layer_elems``."""
        k = len(shard_codes)
        if k != len(shard_scales) or k == 0:
            raise ValueError("need one scales array per codes array")
        if layer_elems > k * shard_elems:
            raise ValueError("layer larger than the shards")
        codes = [_req(c, np.int8) for c in shard_codes]
        scales = [_req(s, np.float32) for s in shard_scales]
        for c, s in zip(codes, scales):
            if c.size < shard_elems or s.size < num_blocks(shard_elems, block):
                raise ValueError("shard buffer too small")
        cptrs = (ctypes.c_void_p * k)(*[c.ctypes.data for c in codes])
        sptrs = (ctypes.c_void_p * k)(*[s.ctypes.data for s in scales])
        out = np.empty(layer_elems, np.uint16)
        self.lib.orc_dequant_gather_layer(cptrs, sptrs, k, shard_elems, block, layer_elems,
                                          _ptr(out))
        return out


    # -- qgZ: int4 gradient quantization and the dequantize-and-reduce ------
    def quantize_blockwise_i4(self, x_f32, block=256):
        """fp32 values -> (packed int4 codes uint8[ceil(n/2)], scales)."""
        x = _req(x_f32, np.float32)
        codes = np.empty((x.size + 1) // 2, np.uint8)
        scales = np.empty(num_blocks(x.size, block), np.float32)
        self.lib.orc_quantize_blockwise_i4(_ptr(x), x.size, block, _ptr(codes), _ptr(scales))
        return codes, scales

    def unpack_i4(self, codes, n):
        codes = _req(codes, np.uint8)
        if codes.size < (n + 1) // 2:
            raise ValueError("too few packed codes")
        out = np.empty(n, np.int8)
        self.lib.orc_unpack_i4(_ptr(codes), n, _ptr(out))
        return out

    def dequant_reduce_i4(self, src_codes, src_scales, n, block, scale_out):
        """Sum over the sources, in order, of the dequantized partition, then
        times scale_out."""
        k = len(src_codes)
        if k != len(src_scales) or k == 0:
            raise ValueError("need one scales array per codes array")
        codes = [_req(c, np.uint8) for c in src_codes]
        scales = [_req(s, np.float32) for s in src_scales]
        for c, s in zip(codes, scales):
            if c.size < (n + 1) // 2 or s.size < num_blocks(n, block):
                raise ValueError("source buffer too small")
        cptrs = (ctypes.c_void_p * k)(*[c.ctypes.data for c in codes])
        sptrs = (ctypes.c_void_p * k)(*[s.ctypes.data for s in scales])
        out = np.empty(n, np.float32)
        self.lib.orc_dequant_reduce_i4(cptrs, sptrs, k, n, block, scale_out, _ptr(out))
        return out


_default = None


def default():
    """The oracle built from the committed source (built on first use)."""
    global _default
    if _default is None:
        if not os.path.exists(_build.LIB):
            _build.build_oracle()
        _default = Oracle(_build.LIB)
    return _default


def bf16_rne(x):
    return default().bf16_rne(x)


def bf16_to_f32(h):
    return default().bf16_to_f32(h)


def adam_step(*args, **kw):
    return default().adam_step(*args, **kw)


def refresh(src):
    return default().refresh(src)


def quantize_blockwise_i8(x_bf16, block=256):
    return default().quantize_blockwise_i8(x_bf16, block)


def dequant_blockwise_i8(codes, scales, block=256):
    return default().dequant_blockwise_i8(codes, scales, block)


def dequant_gather_layer(shard_codes, shard_scales, shard_elems, block, layer_elems):
    return default().dequant_gather_layer(shard_codes, shard_scales, shard_elems, block,
                                          layer_elems)


def quantize_blockwise_i4(x_f32, block=256):
    return default().quantize_blockwise_i4(x_f32, block)


def unpack_i4(codes, n):
    return default().unpack_i4(codes, n)


def dequant_reduce_i4(src_codes, src_scales, n, block, scale_out):
    return default().dequant_reduce_i4(src_codes, src_scales, n, block, scale_out)


# --------------------------------------------------------------------------
# Partition sizes (Eq. 1 and the sentence after it)
# --------------------------------------------------------------------------
def secondary_shard_elems(layer_elems, secondary_world, block=256):
    """|L_second| = N / P' (Eq. 1).  Where P' does not divide N, or the share
    is not a whole number of quantization blocks, the share is rounded up to
    the next whole block and the last shard is zero-padded."""
    share = -(-layer_elems // secondary_world)
    return -(-share // block) * block


def secondary_slice(layer_elems, secondary_world, local_rank, block=256):
    """[begin, end) of the full layer held by ``local_rank``, clipped at N."""
    s = secondary_shard_elems(layer_elems, secondary_world, block)
    begin = min(local_rank * s, layer_elems)
    return begin, min(begin + s, layer_elems)


def primary_slice(layer_elems, world, rank):
    """Rank ``rank``'s contiguous 1/P share of a flat layer (ZeRO-3
    partition); P must divide N."""
    if layer_elems % world:
        raise ValueError("P must divide N for the primary partition")
    n = layer_elems // world
    return rank * n, (rank + 1) * n
