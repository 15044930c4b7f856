"""Python binding of ``libzpp.so`` (the C ABI in ``include/zpp.h``).

Argument marshalling only: every step of the partition path runs in the HIP
kernels of the library.  PyTorch supplies device memory (tensors) and streams;
events are plain HIP events created here.

The library must have been built (``paper_2407_01614_amd.build``); importing
this module fails loudly otherwise.  There is no fallback of any kind.
"""
import ctypes
import os

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libzpp.so")

ZPP_OK, ZPP_EINVAL, ZPP_EALIGN, ZPP_EOVERLAP, ZPP_EHIP = range(5)
MAX_SHARDS = 64
MAX_WAIT_EVENTS = 64

if not os.path.exists(LIB_PATH):
    raise ImportError("libzpp.so is not built (%s); run `python -m paper_2407_01614_amd.build`"
                      % LIB_PATH)

_lib = ctypes.CDLL(LIB_PATH)
_P = ctypes.c_void_p
_sz = ctypes.c_size_t
_u32 = ctypes.c_uint32


class AdamHParams(ctypes.Structure):
    """Mirror of ``zpp_adam_hparams``."""
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("adamw", ctypes.c_int32), ("step", ctypes.c_int64)]


_lib.zpp_adam_partition_step.restype = ctypes.c_int
_lib.zpp_adam_partition_step.argtypes = [_P, _P, _P, _P, _P, _sz, ctypes.POINTER(AdamHParams), _P]
_lib.zpp_adam_step_refresh_quantize.restype = ctypes.c_int
_lib.zpp_adam_step_refresh_quantize.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _sz, _u32,
                                                ctypes.POINTER(AdamHParams), _P, _P, _P]
_lib.zpp_refresh_secondary.restype = ctypes.c_int
_lib.zpp_refresh_secondary.argtypes = [_P, _P, _sz, _P, _P, _P]
_lib.zpp_quantize_blockwise_i8.restype = ctypes.c_int
_lib.zpp_quantize_blockwise_i8.argtypes = [_P, _sz, _u32, _P, _P, _P, _P, _P]
_lib.zpp_refresh_quantize_i8.restype = ctypes.c_int
_lib.zpp_refresh_quantize_i8.argtypes = [_P, _P, _sz, _u32, _P, _P, _P, _P, _P]
_lib.zpp_dequant_gather_layer.restype = ctypes.c_int
_lib.zpp_dequant_gather_layer.argtypes = [_P, _P, _u32, _sz, _u32, _sz, _P, _P, _P, _u32, _P]
_lib.zpp_quantize_blockwise_i4.restype = ctypes.c_int
_lib.zpp_quantize_blockwise_i4.argtypes = [_P, _sz, _u32, _P, _P, _P, _P, _P]
_lib.zpp_dequant_reduce_i4.restype = ctypes.c_int
_lib.zpp_dequant_reduce_i4.argtypes = [_P, _P, _u32, _sz, _u32, ctypes.c_float, _P, _P, _P, _u32,
                                       _P]
_lib.zpp_qgz_receive_adam_step.restype = ctypes.c_int
_lib.zpp_qgz_receive_adam_step.argtypes = [_P, _P, _P, _P, _P, _u32, _u32, ctypes.c_float, _P,
                                           _sz, ctypes.POINTER(AdamHParams), _P, _P, _u32, _P]
_lib.zpp_qgz_receive_step_refresh_quantize.restype = ctypes.c_int
_lib.zpp_qgz_receive_step_refresh_quantize.argtypes = [
    _P, _P, _P, _P, _P, _u32, _u32, ctypes.c_float, _P, _P, _P, _P, _sz, _u32,
    ctypes.POINTER(AdamHParams), _P, _P, _u32, _P]
_lib.zpp_quantize_blockwise_i4_interleaved.restype = ctypes.c_int
_lib.zpp_quantize_blockwise_i4_interleaved.argtypes = [_P, _sz, _u32, _u32, _u32, _P, _P, _P, _P,
                                                       _P]
_lib.zpp_dequant_reduce_i4_interleaved.restype = ctypes.c_int
_lib.zpp_dequant_reduce_i4_interleaved.argtypes = [_P, _P, _u32, _sz, _u32, ctypes.c_float, _P,
                                                   _P, _P, _u32, _P]
_lib.zpp_qgz_receive_adam_step_interleaved.restype = ctypes.c_int
_lib.zpp_qgz_receive_adam_step_interleaved.argtypes = [
    _P, _P, _P, _P, _P, _u32, _u32, ctypes.c_float, _P, _sz, ctypes.POINTER(AdamHParams), _P, _P,
    _u32, _P]
_lib.zpp_qgz_receive_step_refresh_quantize_interleaved.restype = ctypes.c_int
_lib.zpp_qgz_receive_step_refresh_quantize_interleaved.argtypes = [
    _P, _P, _P, _P, _P, _u32, _u32, ctypes.c_float, _P, _P, _P, _P, _sz, _u32,
    ctypes.POINTER(AdamHParams), _P, _P, _u32, _P]
_lib.zpp_status_string.restype = ctypes.c_char_p
_lib.zpp_status_string.argtypes = [ctypes.c_int]
_lib.zpp_last_hip_error.restype = ctypes.c_int
_lib.zpp_last_hip_error.argtypes = []

EXPORTS = ("zpp_adam_partition_step", "zpp_adam_step_refresh_quantize", "zpp_refresh_secondary",
           "zpp_quantize_blockwise_i8", "zpp_refresh_quantize_i8", "zpp_dequant_gather_layer",
           "zpp_quantize_blockwise_i4",
           "zpp_dequant_reduce_i4", "zpp_qgz_receive_adam_step",
           "zpp_qgz_receive_step_refresh_quantize", "zpp_quantize_blockwise_i4_interleaved",
           "zpp_dequant_reduce_i4_interleaved", "zpp_qgz_receive_adam_step_interleaved",
           "zpp_qgz_receive_step_refresh_quantize_interleaved", "zpp_status_string",
           "zpp_last_hip_error")


class ZppError(RuntimeError):
    def __init__(self, status, where=""):
        self.status = status
        msg = _lib.zpp_status_string(status).decode()
        if status == ZPP_EHIP:
            msg += " (hipError_t %d)" % _lib.zpp_last_hip_error()
        super().__init__("%s: %s" % (where, msg) if where else msg)


def _check(status, where):
    if status != ZPP_OK:
        raise ZppError(status, where)


# --------------------------------------------------------------------------
# HIP events and streams (plumbing)
# --------------------------------------------------------------------------
_hip = None


def _hip_lib():
    global _hip
    if _hip is None:
        _hip = ctypes.CDLL("libamdhip64.so")
        _hip.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(_P), ctypes.c_uint]
        _hip.hipEventDestroy.argtypes = [_P]
        _hip.hipEventRecord.argtypes = [_P, _P]
        _hip.hipEventSynchronize.argtypes = [_P]
        _hip.hipEventQuery.argtypes = [_P]
        _hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), _P, _P]
        _hip.hipStreamWaitEvent.argtypes = [_P, _P, ctypes.c_uint]
    return _hip


HIP_EVENT_DEFAULT = 0x0
HIP_EVENT_DISABLE_TIMING = 0x2
HIP_EVENT_DISABLE_SYSTEM_FENCE = 0x20000000


class Event:
    """A HIP event on the current device (timing disabled unless asked).

    `system_fence=False` creates it without the system-scope fence of a
    record: for timing events only, whose records then cost the stream next
    to nothing; such an event must not order memory for the host."""

    def __init__(self, timing=False, system_fence=True):
        h = _hip_lib()
        ev = _P()
        flags = HIP_EVENT_DEFAULT if timing else HIP_EVENT_DISABLE_TIMING
        if not system_fence:
            flags |= HIP_EVENT_DISABLE_SYSTEM_FENCE
        err = h.hipEventCreateWithFlags(ctypes.byref(ev), flags)
        if err:
            raise RuntimeError("hipEventCreateWithFlags failed: %d" % err)
        self.handle = ev.value

    def record(self, stream=None):
        err = _hip_lib().hipEventRecord(self.handle, stream_handle(stream))
        if err:
            raise RuntimeError("hipEventRecord failed: %d" % err)
        return self

    def synchronize(self):
        err = _hip_lib().hipEventSynchronize(self.handle)
        if err:
            raise RuntimeError("hipEventSynchronize failed: %d" % err)

    def query(self):
        """True once every piece of work recorded before the event is done."""
        return _hip_lib().hipEventQuery(self.handle) == 0

    def elapsed_ms(self, end):
        ms = ctypes.c_float()
        err = _hip_lib().hipEventElapsedTime(ctypes.byref(ms), self.handle, end.handle)
        if err:
            raise RuntimeError("hipEventElapsedTime failed: %d" % err)
        return ms.value

    def __del__(self):
        h = self.__dict__.get("handle")
        if h and _hip is not None:
            try:
                _hip.hipEventDestroy(h)
            except Exception:
                pass


def stream_wait(stream, event):
    """Make `stream` wait on the device for `event` (hipStreamWaitEvent)."""
    err = _hip_lib().hipStreamWaitEvent(stream_handle(stream), _event_handle(event), 0)
    if err:
        raise RuntimeError("hipStreamWaitEvent failed: %d" % err)


def stream_handle(stream):
    """Raw hipStream_t of a torch stream, an int handle, or None (the current
    torch stream of the current device)."""
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    if stream.device.index != torch.cuda.current_device():
        raise ValueError("stream of %s, not of the current device cuda:%d"
                         % (stream.device, torch.cuda.current_device()))
    return stream.cuda_stream


def _event_handle(ev):
    if ev is None:
        return None
    if isinstance(ev, Event):
        return ev.handle
    if isinstance(ev, int):
        return ev
    raise TypeError("expected zpp.Event, int handle or None")


# --------------------------------------------------------------------------
# Tensor checks (marshalling)
# --------------------------------------------------------------------------
def _dev(t, dtypes, name):
    if not isinstance(t, torch.Tensor):
        raise TypeError("%s must be a torch.Tensor" % name)
    if not t.is_cuda:
        raise ValueError("%s must be on the GPU" % name)
    if t.device.index != torch.cuda.current_device():
        # the library launches on the current device; a pointer into another
        # device's memory would be dereferenced there
        raise ValueError("%s is on %s, not on the current device cuda:%d"
                         % (name, t.device, torch.cuda.current_device()))
    if t.dtype not in dtypes:
        raise TypeError("%s: dtype %s not in %s" % (name, t.dtype, dtypes))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)
    return t


_F32 = (torch.float32,)
_BF16 = (torch.bfloat16, torch.int16, torch.uint16)
_I8 = (torch.int8,)
_U8 = (torch.uint8, torch.int8)


# --------------------------------------------------------------------------
# The four calls
# --------------------------------------------------------------------------
def adam_partition_step(master, exp_avg, exp_avg_sq, grad, primary_bf16, *, lr, beta1, beta2,
                        eps, weight_decay, step, adamw=True, n=None, stream=None):
    """zpp_adam_partition_step over the first ``n`` elements (default: all)."""
    for t, name in ((master, "master"), (exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq"),
                    (grad, "grad")):
        _dev(t, _F32, name)
    _dev(primary_bf16, _BF16, "primary_bf16")
    if n is None:
        n = master.numel()
    if any(t.numel() < n for t in (master, exp_avg, exp_avg_sq, grad, primary_bf16)):
        raise ValueError("a buffer holds fewer than n elements")
    hp = AdamHParams(lr, beta1, beta2, eps, weight_decay, 1 if adamw else 0, int(step))
    st = _lib.zpp_adam_partition_step(master.data_ptr(), exp_avg.data_ptr(),
                                      exp_avg_sq.data_ptr(), grad.data_ptr(),
                                      primary_bf16.data_ptr(), n, ctypes.byref(hp),
                                      stream_handle(stream))
    _check(st, "zpp_adam_partition_step")


def adam_step_refresh_quantize(master, exp_avg, exp_avg_sq, grad, primary_bf16, secondary_bf16,
                               codes, scales, *, lr, beta1, beta2, eps, weight_decay, step,
                               adamw=True, block=256, n=None, stream=None, wait_before=None,
                               done_after=None):
    """zpp_adam_step_refresh_quantize: the partition step, the secondary copy
    (``secondary_bf16`` may be None) and its int8 quantization in one pass."""
    for t, name in ((master, "master"), (exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq"),
                    (grad, "grad"), (scales, "scales")):
        _dev(t, _F32, name)
    _dev(primary_bf16, _BF16, "primary_bf16")
    if secondary_bf16 is not None:
        _dev(secondary_bf16, _BF16, "secondary_bf16")
    _dev(codes, _I8, "codes")
    if n is None:
        n = master.numel()
    bufs = [master, exp_avg, exp_avg_sq, grad, primary_bf16, codes]
    if secondary_bf16 is not None:
        bufs.append(secondary_bf16)
    if any(t.numel() < n for t in bufs) or scales.numel() < num_blocks(n, block):
        raise ValueError("a buffer is too small for n = %d" % n)
    hp = AdamHParams(lr, beta1, beta2, eps, weight_decay, 1 if adamw else 0, int(step))
    st = _lib.zpp_adam_step_refresh_quantize(
        master.data_ptr(), exp_avg.data_ptr(), exp_avg_sq.data_ptr(), grad.data_ptr(),
        primary_bf16.data_ptr(), secondary_bf16.data_ptr() if secondary_bf16 is not None else None,
        codes.data_ptr(), scales.data_ptr(), n, block, ctypes.byref(hp), stream_handle(stream),
        _event_handle(wait_before), _event_handle(done_after))
    _check(st, "zpp_adam_step_refresh_quantize")


def refresh_secondary(secondary_bf16, src_bf16, count=None, *, stream=None, wait_before=None,
                      done_after=None):
    """zpp_refresh_secondary: copy ``count`` bf16 (default: all of src)."""
    _dev(secondary_bf16, _BF16, "secondary_bf16")
    _dev(src_bf16, _BF16, "src_bf16")
    if count is None:
        count = src_bf16.numel()
    if secondary_bf16.numel() < count or src_bf16.numel() < count:
        raise ValueError("a buffer holds fewer than count elements")
    st = _lib.zpp_refresh_secondary(secondary_bf16.data_ptr(), src_bf16.data_ptr(), count,
                                    stream_handle(stream), _event_handle(wait_before),
                                    _event_handle(done_after))
    _check(st, "zpp_refresh_secondary")


def num_blocks(n, block):
    """Blocks of `block` elements covering n; 0 for a block size the library
    rejects anyway (it reports that as ZPP_EINVAL)."""
    return (n + block - 1) // block if block > 0 else 0


def quantize_blockwise_i8(src_bf16, codes, scales, *, block=256, n=None, stream=None,
                          wait_before=None, done_after=None):
    """zpp_quantize_blockwise_i8 over the first ``n`` elements of src."""
    _dev(src_bf16, _BF16, "src_bf16")
    _dev(codes, _I8, "codes")
    _dev(scales, _F32, "scales")
    if n is None:
        n = src_bf16.numel()
    if src_bf16.numel() < n or codes.numel() < n or scales.numel() < num_blocks(n, block):
        raise ValueError("a buffer is too small for n = %d" % n)
    st = _lib.zpp_quantize_blockwise_i8(src_bf16.data_ptr(), n, block, codes.data_ptr(),
                                        scales.data_ptr(), stream_handle(stream),
                                        _event_handle(wait_before), _event_handle(done_after))
    _check(st, "zpp_quantize_blockwise_i8")


def refresh_quantize_i8(secondary_bf16, src_bf16, codes, scales, *, block=256, n=None,
                        stream=None, wait_before=None, done_after=None):
    """zpp_refresh_quantize_i8 over the first ``n`` elements of src: the
    secondary refresh and its quantization in one pass."""
    _dev(secondary_bf16, _BF16, "secondary_bf16")
    _dev(src_bf16, _BF16, "src_bf16")
    _dev(codes, _I8, "codes")
    _dev(scales, _F32, "scales")
    if n is None:
        n = src_bf16.numel()
    if (src_bf16.numel() < n or secondary_bf16.numel() < n or codes.numel() < n
            or scales.numel() < num_blocks(n, block)):
        raise ValueError("a buffer is too small for n = %d" % n)
    st = _lib.zpp_refresh_quantize_i8(secondary_bf16.data_ptr(), src_bf16.data_ptr(), n, block,
                                      codes.data_ptr(), scales.data_ptr(), stream_handle(stream),
                                      _event_handle(wait_before), _event_handle(done_after))
    _check(st, "zpp_refresh_quantize_i8")


def dequant_gather_layer(shard_codes, shard_scales, shard_elems, layer_elems, out_bf16, *,
                         block=256, stream=None, wait_events=(), done_after=None):
    """zpp_dequant_gather_layer over P' = len(shard_codes) shards."""
    k = len(shard_codes)
    if k != len(shard_scales):
        raise ValueError("one scales tensor per codes tensor")
    if not 1 <= k <= MAX_SHARDS:
        raise ValueError("1..%d shards" % MAX_SHARDS)
    for j in range(k):
        _dev(shard_codes[j], _I8, "shard_codes[%d]" % j)
        _dev(shard_scales[j], _F32, "shard_scales[%d]" % j)
        if (shard_codes[j].numel() < shard_elems
                or shard_scales[j].numel() < num_blocks(shard_elems, block)):
            raise ValueError("shard %d buffers too small" % j)
    _dev(out_bf16, _BF16, "out_bf16")
    if out_bf16.numel() < layer_elems:
        raise ValueError("out holds fewer than layer_elems elements")
    cptrs = (_P * k)(*[c.data_ptr() for c in shard_codes])
    sptrs = (_P * k)(*[s.data_ptr() for s in shard_scales])
    waits = [_event_handle(e) for e in wait_events]
    warr = (_P * max(1, len(waits)))(*waits) if waits else None
    st = _lib.zpp_dequant_gather_layer(cptrs, sptrs, k, shard_elems, block, layer_elems,
                                       out_bf16.data_ptr(), stream_handle(stream), warr,
                                       len(waits), _event_handle(done_after))
    _check(st, "zpp_dequant_gather_layer")


def quantize_blockwise_i4(src, codes, scales, *, block=256, n=None, stream=None,
                          wait_before=None, done_after=None):
    """zpp_quantize_blockwise_i4 of the first ``n`` fp32 values of src."""
    _dev(src, _F32, "src")
    _dev(codes, _U8, "codes")
    _dev(scales, _F32, "scales")
    if n is None:
        n = src.numel()
    if src.numel() < n or codes.numel() < (n + 1) // 2 or scales.numel() < num_blocks(n, block):
        raise ValueError("a buffer is too small for n = %d" % n)
    st = _lib.zpp_quantize_blockwise_i4(src.data_ptr(), n, block, codes.data_ptr(),
                                        scales.data_ptr(), stream_handle(stream),
                                        _event_handle(wait_before), _event_handle(done_after))
    _check(st, "zpp_quantize_blockwise_i4")


def dequant_reduce_i4(src_codes, src_scales, n, out, *, block=256, scale_out=1.0, stream=None,
                      wait_events=(), done_after=None):
    """zpp_dequant_reduce_i4 over len(src_codes) sources into out[:n]."""
    k = len(src_codes)
    if k != len(src_scales) or not 1 <= k <= MAX_SHARDS:
        raise ValueError("1..%d sources, one scales tensor each" % MAX_SHARDS)
    for q in range(k):
        _dev(src_codes[q], _U8, "src_codes[%d]" % q)
        _dev(src_scales[q], _F32, "src_scales[%d]" % q)
        if src_codes[q].numel() < (n + 1) // 2 or src_scales[q].numel() < num_blocks(n, block):
            raise ValueError("source %d buffers too small" % q)
    _dev(out, _F32, "out")
    if out.numel() < n:
        raise ValueError("out holds fewer than n elements")
    cptrs = (_P * k)(*[c.data_ptr() for c in src_codes])
    sptrs = (_P * k)(*[x.data_ptr() for x in src_scales])
    waits = [_event_handle(e) for e in wait_events]
    warr = (_P * len(waits))(*waits) if waits else None
    st = _lib.zpp_dequant_reduce_i4(cptrs, sptrs, k, n, block, scale_out, out.data_ptr(),
                                    stream_handle(stream), warr, len(waits),
                                    _event_handle(done_after))
    _check(st, "zpp_dequant_reduce_i4")


def qgz_receive_adam_step(master, exp_avg, exp_avg_sq, src_codes, src_scales, primary_bf16, *,
                          lr, beta1, beta2, eps, weight_decay, step, adamw=True, block=256,
                          scale_out=1.0, n=None, stream=None, wait_events=(), done_after=None):
    """zpp_qgz_receive_adam_step: the partition step with its gradient taken
    from len(src_codes) int4 copies (the mean when scale_out = 1/len)."""
    for t, name in ((master, "master"), (exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq")):
        _dev(t, _F32, name)
    _dev(primary_bf16, _BF16, "primary_bf16")
    k = len(src_codes)
    if k != len(src_scales) or not 1 <= k <= MAX_SHARDS:
        raise ValueError("1..%d sources, one scales tensor each" % MAX_SHARDS)
    if n is None:
        n = master.numel()
    for q in range(k):
        _dev(src_codes[q], _U8, "src_codes[%d]" % q)
        _dev(src_scales[q], _F32, "src_scales[%d]" % q)
        if src_codes[q].numel() < (n + 1) // 2 or src_scales[q].numel() < num_blocks(n, block):
            raise ValueError("source %d buffers too small" % q)
    if any(t.numel() < n for t in (master, exp_avg, exp_avg_sq, primary_bf16)):
        raise ValueError("a buffer holds fewer than n elements")
    cptrs = (_P * k)(*[c.data_ptr() for c in src_codes])
    sptrs = (_P * k)(*[x.data_ptr() for x in src_scales])
    waits = [_event_handle(e) for e in wait_events]
    warr = (_P * len(waits))(*waits) if waits else None
    hp = AdamHParams(lr, beta1, beta2, eps, weight_decay, 1 if adamw else 0, int(step))
    st = _lib.zpp_qgz_receive_adam_step(master.data_ptr(), exp_avg.data_ptr(),
                                        exp_avg_sq.data_ptr(), cptrs, sptrs, k, block, scale_out,
                                        primary_bf16.data_ptr(), n, ctypes.byref(hp),
                                        stream_handle(stream), warr, len(waits),
                                        _event_handle(done_after))
    _check(st, "zpp_qgz_receive_adam_step")


def qgz_receive_step_refresh_quantize(master, exp_avg, exp_avg_sq, src_codes, src_scales,
                                      primary_bf16, secondary_bf16, codes, scales, *, lr, beta1,
                                      beta2, eps, weight_decay, step, adamw=True, grad_block=256,
                                      block=256, scale_out=1.0, n=None, stream=None,
                                      wait_events=(), done_after=None):
    """zpp_qgz_receive_step_refresh_quantize: the receive step, the secondary
    copy (``secondary_bf16`` may be None) and its int8 quantization in one
    pass."""
    for t, name in ((master, "master"), (exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq"),
                    (scales, "scales")):
        _dev(t, _F32, name)
    _dev(primary_bf16, _BF16, "primary_bf16")
    if secondary_bf16 is not None:
        _dev(secondary_bf16, _BF16, "secondary_bf16")
    _dev(codes, _I8, "codes")
    k = len(src_codes)
    if k != len(src_scales) or not 1 <= k <= MAX_SHARDS:
        raise ValueError("1..%d sources, one scales tensor each" % MAX_SHARDS)
    if n is None:
        n = master.numel()
    for q in range(k):
        _dev(src_codes[q], _U8, "src_codes[%d]" % q)
        _dev(src_scales[q], _F32, "src_scales[%d]" % q)
        if (src_codes[q].numel() < (n + 1) // 2
                or src_scales[q].numel() < num_blocks(n, grad_block)):
            raise ValueError("source %d buffers too small" % q)
    bufs = [master, exp_avg, exp_avg_sq, primary_bf16, codes]
    if secondary_bf16 is not None:
        bufs.append(secondary_bf16)
    if any(t.numel() < n for t in bufs) or scales.numel() < num_blocks(n, block):
        raise ValueError("a buffer is too small for n = %d" % n)
    cptrs = (_P * k)(*[c.data_ptr() for c in src_codes])
    sptrs = (_P * k)(*[x.data_ptr() for x in src_scales])
    waits = [_event_handle(e) for e in wait_events]
    warr = (_P * len(waits))(*waits) if waits else None
    hp = AdamHParams(lr, beta1, beta2, eps, weight_decay, 1 if adamw else 0, int(step))
    st = _lib.zpp_qgz_receive_step_refresh_quantize(
        master.data_ptr(), exp_avg.data_ptr(), exp_avg_sq.data_ptr(), cptrs, sptrs, k, grad_block,
        scale_out, primary_bf16.data_ptr(),
        secondary_bf16.data_ptr() if secondary_bf16 is not None else None, codes.data_ptr(),
        scales.data_ptr(), n, block, ctypes.byref(hp), stream_handle(stream), warr, len(waits),
        _event_handle(done_after))
    _check(st, "zpp_qgz_receive_step_refresh_quantize")


# --------------------------------------------------------------------------
# The qgZ receive buffer interleaved (layout in include/zpp.h)
# --------------------------------------------------------------------------
def interleaved_sizes(n, block, num_src):
    """(code bytes, scale count) of an interleaved receive buffer of num_src
    int4 copies of n elements in blocks of `block`."""
    nb = num_blocks(n, block)
    return nb * num_src * (block // 2), nb * num_src


def _interleaved_inputs(codes, scales, n, block, num_src):
    _dev(codes, _U8, "codes")
    _dev(scales, _F32, "scales")
    if not 1 <= num_src <= MAX_SHARDS:
        raise ValueError("1..%d sources" % MAX_SHARDS)
    nc, ns = interleaved_sizes(n, block, num_src)
    if codes.numel() < nc or scales.numel() < ns:
        raise ValueError("the interleaved buffer is too small for n = %d, %d sources" % (n, num_src))


def quantize_blockwise_i4_interleaved(src, codes, scales, *, source, num_src, block=256, n=None,
                                      stream=None, wait_before=None, done_after=None):
    """zpp_quantize_blockwise_i4_interleaved: source `source` of num_src."""
    _dev(src, _F32, "src")
    if n is None:
        n = src.numel()
    if src.numel() < n:
        raise ValueError("src holds fewer than n elements")
    _interleaved_inputs(codes, scales, n, block, num_src)
    st = _lib.zpp_quantize_blockwise_i4_interleaved(
        src.data_ptr(), n, block, source, num_src, codes.data_ptr(), scales.data_ptr(),
        stream_handle(stream), _event_handle(wait_before), _event_handle(done_after))
    _check(st, "zpp_quantize_blockwise_i4_interleaved")


def dequant_reduce_i4_interleaved(codes, scales, num_src, n, out, *, block=256, scale_out=1.0,
                                  stream=None, wait_events=(), done_after=None):
    """zpp_dequant_reduce_i4_interleaved: the num_src int4 copies of one
    interleaved receive buffer reduced into out[:n]."""
    _interleaved_inputs(codes, scales, n, block, num_src)
    _dev(out, _F32, "out")
    if out.numel() < n:
        raise ValueError("out holds fewer than n elements")
    waits = [_event_handle(e) for e in wait_events]
    warr = (_P * len(waits))(*waits) if waits else None
    st = _lib.zpp_dequant_reduce_i4_interleaved(
        codes.data_ptr(), scales.data_ptr(), num_src, n, block, scale_out, out.data_ptr(),
        stream_handle(stream), warr, len(waits), _event_handle(done_after))
    _check(st, "zpp_dequant_reduce_i4_interleaved")


def qgz_receive_adam_step_interleaved(master, exp_avg, exp_avg_sq, codes, scales, num_src,
                                      primary_bf16, *, lr, beta1, beta2, eps, weight_decay,
                                      step, adamw=True, block=256, scale_out=1.0, n=None,
                                      stream=None, wait_events=(), done_after=None):
    """zpp_qgz_receive_adam_step_interleaved: the receive step from one
    interleaved buffer of num_src int4 copies."""
    for t, name in ((master, "master"), (exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq")):
        _dev(t, _F32, name)
    _dev(primary_bf16, _BF16, "primary_bf16")
    if n is None:
        n = master.numel()
    if any(t.numel() < n for t in (master, exp_avg, exp_avg_sq, primary_bf16)):
        raise ValueError("a buffer holds fewer than n elements")
    _interleaved_inputs(codes, scales, n, block, num_src)
    waits = [_event_handle(e) for e in wait_events]
    warr = (_P * len(waits))(*waits) if waits else None
    hp = AdamHParams(lr, beta1, beta2, eps, weight_decay, 1 if adamw else 0, int(step))
    st = _lib.zpp_qgz_receive_adam_step_interleaved(
        master.data_ptr(), exp_avg.data_ptr(), exp_avg_sq.data_ptr(), codes.data_ptr(),
        scales.data_ptr(), num_src, block, scale_out, primary_bf16.data_ptr(), n,
        ctypes.byref(hp), stream_handle(stream), warr, len(waits), _event_handle(done_after))
    _check(st, "zpp_qgz_receive_adam_step_interleaved")


def qgz_receive_step_refresh_quantize_interleaved(
        master, exp_avg, exp_avg_sq, src_codes, src_scales, num_src, primary_bf16,
        secondary_bf16, codes, scales, *, lr, beta1, beta2, eps, weight_decay, step, adamw=True,
        grad_block=256, block=256, scale_out=1.0, n=None, stream=None, wait_events=(),
        done_after=None):
    """zpp_qgz_receive_step_refresh_quantize_interleaved: the single pass from
    one interleaved buffer of num_src int4 copies."""
    for t, name in ((master, "master"), (exp_avg, "exp_avg"), (exp_avg_sq, "exp_avg_sq"),
                    (scales, "scales")):
        _dev(t, _F32, name)
    _dev(primary_bf16, _BF16, "primary_bf16")
    if secondary_bf16 is not None:
        _dev(secondary_bf16, _BF16, "secondary_bf16")
    _dev(codes, _I8, "codes")
    if n is None:
        n = master.numel()
    bufs = [master, exp_avg, exp_avg_sq, primary_bf16, codes]
    if secondary_bf16 is not None:
        bufs.append(secondary_bf16)
    if any(t.numel() < n for t in bufs) or scales.numel() < num_blocks(n, block):
        raise ValueError("a buffer is too small for n = %d" % n)
    _interleaved_inputs(src_codes, src_scales, n, grad_block, num_src)
    waits = [_event_handle(e) for e in wait_events]
    warr = (_P * len(waits))(*waits) if waits else None
    hp = AdamHParams(lr, beta1, beta2, eps, weight_decay, 1 if adamw else 0, int(step))
    st = _lib.zpp_qgz_receive_step_refresh_quantize_interleaved(
        master.data_ptr(), exp_avg.data_ptr(), exp_avg_sq.data_ptr(), src_codes.data_ptr(),
        src_scales.data_ptr(), num_src, grad_block, scale_out, primary_bf16.data_ptr(),
        secondary_bf16.data_ptr() if secondary_bf16 is not None else None, codes.data_ptr(),
        scales.data_ptr(), n, block, ctypes.byref(hp), stream_handle(stream), warr, len(waits),
        _event_handle(done_after))
    _check(st, "zpp_qgz_receive_step_refresh_quantize_interleaved")


# --------------------------------------------------------------------------
# Raw entry (pointers and sizes, no tensor checks) for ABI tests
# --------------------------------------------------------------------------
raw = _lib
