"""Benchmark of one rank's partition path on one MI355X.

A step is one pass of the whole path over one rank's state: the Adam
partition step, the secondary refresh, its int8 quantization, and the
dequant-gather of the layers of the backward pass from the P' node-local
secondary shards (one layer for the Llama-2 workloads; Falcon-40B's step
gathers its 60 layers).  The headline runs these kernels in that order on one
HIP stream, so the stream order is the ordering fix of the paper: the gather
cannot start before the quantization of the copy it reads has finished.

Prints ONE JSON line.  `value` is the algorithmic HBM bytes of all kernels of
a step divided by the measured wall time per step (GB/s), with every input
resident in HBM.  The roofline entry is the dominant kernel's (the Adam
step): its algorithmic bytes over its mean launch duration in those same K
timed steps, each Adam launch bracketed by a HIP timing-event pair on its
stream (events without the system-scope fence, whose records cost the step
next to nothing).  The per-kernel table comes from a second run of K steps
with a pair around every kernel.  Beside it: the same step on three
streams ordered by events (with and without one step's gather overlapping the
next step's Adam), the fused step + refresh + quantize kernel in place of the
three separate ones, the time per step with the gather ordered by a device
event wait (the fix), by a host-side wait, or not at all (stock hpZ, racy:
timing only), the step with the refresh and its quantization as one pass,
the qgZ gradient side, the step preceded by the qgZ receive
of eight int4 copies delivered into one interleaved receive buffer (as its
own kernel, fused into the partition step, and inside the single pass of
step, refresh and quantization), the forward AllGather(L, P) with qwZ as one
GPU carries it (the P ranks' bf16 primary slices int8-quantized, then the
layer gathered from them), the HBM ceilings of this GPU (read-only,
write-only and copy streams, each kernel reported as a fraction of the copy)
and, for context, PyTorch's fused AdamW on a partition of the same size.
The CPU baseline times the plain CPU oracle on a bounded sample of the same
workload on this host.

    python bench.py [--gpus 1] [--steps 200] [--warmup 10] [--workload llama-2-13b]
"""
import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0  # MI355X HBM3E, AMD's published figure
METRIC = "achieved HBM GB/s (and % of peak) for partition step+refresh and dequant-gather"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=10)
    from paper_2407_01614_amd.workloads import WORKLOADS
    # a step stores its gather shards in the rank's own partition; the tiny
    # configuration (4 ranks of 1 Mi elements gathering a 4 Mi layer from 2
    # shards) does not fit that and is covered by the parity tests instead
    benchable = [k for k, w in WORKLOADS.items() if w.distinct_layers * w.shard_elems <= w.n]
    ap.add_argument("--workload", default="llama-2-13b", choices=benchable)
    ap.add_argument("--cpu-sample", type=float, default=1.0,
                    help="fraction of the workload the CPU oracle is timed on (0 = skip)")
    ap.add_argument("--cpu-steps", type=int, default=2,
                    help="consecutive steps the CPU oracle is timed over")
    ap.add_argument("--cpu-other", type=int, default=1,
                    help="also time the CPU oracle at the other workloads (1) or not (0)")
    ap.add_argument("--sustain-s", type=float, default=10.0,
                    help="seconds of back-to-back headline steps after the timed ones, reported "
                         "as `sustained` (0 = skip)")
    ap.add_argument("--traffic", default=os.path.join(ROOT, "profiles", "traffic.json"),
                    help="measured HBM bytes per launch from rocprofv3 counters, if present")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run a plain 1 GiB device copy 5 times, the known-size reference "
                         "that scales rocprofv3's FETCH_SIZE / WRITE_SIZE counters")
    ap.add_argument("--no-clock-query", action="store_true",
                    help="do not start the amd-smi child that reports the clock policy (under "
                         "rocprofv3 --pmc the profiler's preloaded library initialises the GPU in "
                         "every child process, before amd-smi's interpreter is started)")
    return ap.parse_args()


# The sources each kernel is built from: a counter figure in the traffic file
# is reported only while their digest still matches.
_COMMON = ["zpp_device.h", "zpp_launch.h"]
TRAFFIC_SOURCES = {
    "adam": ["adam.hip", "zpp_adam.h"] + _COMMON,
    "refresh": ["refresh.hip"] + _COMMON,
    "quant": ["quant.hip", "zpp_quant.h", "zpp_chunk.h"] + _COMMON,
    "refresh_quant": ["quant.hip", "zpp_quant.h", "zpp_chunk.h"] + _COMMON,
    "gather": ["gather.hip"] + _COMMON,
    "fused": ["fused.hip", "zpp_adam.h", "zpp_quant.h", "zpp_i4grad.h", "zpp_chunk.h"] + _COMMON,
    "quant_i4": ["qgz.hip", "zpp_quant.h", "zpp_i4grad.h", "zpp_chunk.h"] + _COMMON,
    "reduce_i4": ["qgz.hip", "zpp_i4grad.h", "zpp_quant.h", "zpp_chunk.h"] + _COMMON,
    "receive_adam": ["receive_adam.hip", "zpp_adam.h", "zpp_quant.h", "zpp_i4grad.h",
                     "zpp_chunk.h"] + _COMMON,
    "fused_receive": ["fused.hip", "zpp_adam.h", "zpp_quant.h", "zpp_i4grad.h",
                      "zpp_chunk.h"] + _COMMON,
}


def source_digest(sources):
    """The first 16 hex digits of the SHA-256 of the named csrc files."""
    h = hashlib.sha256()
    for fn in sources:
        with open(os.path.join(ROOT, "paper_2407_01614_amd", "csrc", fn), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def measured_traffic(path, workload, kernel, sources):
    """HBM bytes per launch of `kernel` measured with rocprofv3 FETCH_SIZE /
    WRITE_SIZE (scaled by a plain copy of known size), or None when absent or
    when the kernel's sources changed since the counters were taken."""
    if not os.path.exists(path):
        return None
    with open(path) as f:
        tr = json.load(f)
    entry = tr.get("kernels", {}).get(kernel)
    if tr.get("workload") != workload or entry is None:
        return None
    if source_digest(sources) != entry.get("source_digest"):
        return None
    return round(entry["bytes_per_launch"])


def kernel_table(kb, times, copy_gbps=None):
    """Per kernel: algorithmic bytes, launch durations (mean, median, min),
    GB/s at the median duration (one launch delayed by the host, e.g. a
    descheduled thread while the stream had run dry, moves the mean but not
    the median), the fraction of the HBM peak and, given the copy ceiling
    measured in the same run, the fraction of that."""
    out = {}
    for k in kb:
        ts = sorted(times[k])
        mean = sum(ts) / len(ts)
        med = ts[len(ts) // 2]
        gbps = kb[k] / (med * 1e-3) / 1e9
        out[k] = {"bytes": kb[k], "mean_us": round(mean * 1e3, 2),
                  "median_us": round(med * 1e3, 2), "min_us": round(ts[0] * 1e3, 2),
                  "GB/s": round(gbps, 1), "frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4)}
        if copy_gbps:
            out[k]["frac_of_copy_ceiling"] = round(gbps / copy_gbps, 4)
    return out


def forward_slices(wl, stream):
    """The forward AllGather(L, P) with qwZ up to the exchange: a layer of
    N bf16 weights ~ N(0, 0.02) split into the P ranks' primary slices of
    s = ceil(N/P) rounded up to the block (the last zero-padded), each slice
    quantized by zpp_quantize_blockwise_i8 as its rank does before the
    exchange.  Returns s, the weights, the codes and the scales."""
    import torch
    from paper_2407_01614_amd import synth, zpp
    from paper_2407_01614_amd.workloads import secondary_elems
    P, N, B = wl.world, wl.layer_elems, wl.block
    s = secondary_elems(N, P, B)
    w = synth.device_bf16_weights(P * s, wl.cfg_id, rank=1000)
    w[N:] = 0
    codes = [torch.empty(s, dtype=torch.int8, device="cuda") for _ in range(P)]
    scales = [torch.empty(s // B, dtype=torch.float32, device="cuda") for _ in range(P)]
    for j in range(P):
        zpp.quantize_blockwise_i8(w[j * s:(j + 1) * s], codes[j], scales[j], block=B,
                                  stream=stream)
    return s, w, codes, scales


def forward_gather_measure(wl, reps):
    """The forward AllGather(L, P) with qwZ, as far as one GPU carries it:
    the P ranks' primary slices of a layer, int8-quantized each by the
    library (forward_slices, not timed), then the layer assembled from all P
    slices by the same dequant-gather kernel over P shards (64 at most per
    call; a larger world takes several calls, each writing its part of the
    layer).  The exchange that brings the slices from the other nodes needs
    more GPUs.  Timed with events over `reps` launches (GB/s at the median);
    the quantization of one slice, what each rank does before the exchange,
    is timed too."""
    import torch
    from paper_2407_01614_amd import zpp
    from paper_2407_01614_amd.workloads import bytes_gather, bytes_quant
    P, N, B = wl.world, wl.layer_elems, wl.block
    stream = torch.cuda.Stream()
    s, w, codes, scales = forward_slices(wl, stream)
    qevs = []
    for _ in range(reps):
        a, b = zpp.Event(timing=True), zpp.Event(timing=True)
        a.record(stream)
        zpp.quantize_blockwise_i8(w[:s], codes[0], scales[0], block=B, stream=stream)
        b.record(stream)
        qevs.append((a, b))
    out = torch.empty(N, dtype=torch.int16, device="cuda")
    G = zpp.MAX_SHARDS
    groups = []
    for g0 in range(0, P, G):
        part = min(N - g0 * s, min(G, P - g0) * s)
        if part > 0:
            # the checked binding once (tensor shapes, dtypes, devices) ...
            zpp.dequant_gather_layer(codes[g0:g0 + G], scales[g0:g0 + G], s, part,
                                     out[g0 * s:], block=B, stream=stream)
            k = min(G, P - g0)
            groups.append(((ctypes.c_void_p * k)(*[c.data_ptr() for c in codes[g0:g0 + k]]),
                           (ctypes.c_void_p * k)(*[x.data_ptr() for x in scales[g0:g0 + k]]),
                           k, part, out[g0 * s:].data_ptr()))
    sh = ctypes.c_void_p(zpp.stream_handle(stream))

    def once():
        # ... then the C entry point straight from prepared pointer arrays, so
        # that marshalling 64 tensors per call does not leave the GPU waiting
        # for the next launch inside a timed interval
        for cp, sp, k, part, optr in groups:
            st = zpp.raw.zpp_dequant_gather_layer(cp, sp, k, s, B, part, optr, sh, None, 0, None)
            if st != zpp.ZPP_OK:
                raise zpp.ZppError(st, "zpp_dequant_gather_layer")

    evs = []
    for _ in range(reps):
        a, b = zpp.Event(timing=True), zpp.Event(timing=True)
        a.record(stream)
        once()
        b.record(stream)
        evs.append((a, b))
    torch.cuda.synchronize()
    ts = sorted(a.elapsed_ms(b) for a, b in evs)
    mean, med = sum(ts) / len(ts), ts[len(ts) // 2]
    qmean = sum(a.elapsed_ms(b) for a, b in qevs) / len(qevs)
    nbytes = bytes_gather(s, P, N, B)
    gbps = nbytes / (med * 1e-3) / 1e9
    del w, codes, scales, out
    return {"ranks": P, "slice_elems": s, "layer_elems": N, "launches_per_gather": -(-P // G),
            "codes": "each slice int8-quantized by the library from bf16 weights ~ N(0, 0.02)",
            "bytes": nbytes, "mean_us": round(mean * 1e3, 2), "median_us": round(med * 1e3, 2),
            "GB/s": round(gbps, 1),
            "frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4),
            "quantize_one_slice": {"bytes": bytes_quant(s, B), "mean_us": round(qmean * 1e3, 2)}}


def torch_adamw_context(wl, reps):
    """Context, not the product path: PyTorch's own fused AdamW step
    (torch.optim.AdamW(fused=True)) on a partition of the same size, followed
    by the bf16 copy of the weights that the partition step emits in the same
    pass; timed with events over `reps` steps.  Same hyperparameters and the
    same 30 B per element of algorithmic traffic."""
    import torch
    from paper_2407_01614_amd import synth
    p = torch.nn.Parameter(synth.device_normal_f32(wl.n, synth.WEIGHT_STD, wl.cfg_id,
                                                   synth.KIND_MASTER))
    p.grad = synth.device_normal_f32(wl.n, synth.GRAD_STD, wl.cfg_id, synth.KIND_GRAD)
    out = torch.empty(wl.n, dtype=torch.bfloat16, device="cuda")
    opt = torch.optim.AdamW([p], lr=wl.lr, betas=(wl.beta1, wl.beta2), eps=wl.eps,
                            weight_decay=wl.weight_decay, fused=True)

    def step():
        opt.step()
        out.copy_(p.detach())

    for _ in range(3):
        step()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(reps)]
    for a, b in evs:
        a.record()
        step()
        b.record()
    torch.cuda.synchronize()
    ms = sum(a.elapsed_time(b) for a, b in evs) / reps
    gbps = 30.0 * wl.n / (ms * 1e-3) / 1e9
    del opt, p, out
    torch.cuda.empty_cache()
    return {"what": "torch.optim.AdamW(fused=True).step() + bf16 copy of the weights, same "
                    "partition and hyperparameters (context, not the product path)",
            "ms_per_step": round(ms, 4), "GB/s": round(gbps, 1),
            "frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4)}


CEILING_LIB = os.path.join(ROOT, "paper_2407_01614_amd", "libzpp_ceiling.so")


def ceilings(reps=20):
    """The HBM ceilings of this GPU, measured in this run on 1 GiB streams
    (include/zpp_ceiling.h: 16-byte non-temporal accesses in the launch
    shapes that stream fastest): read-only, write-only and copy; beside
    them the runtime's device-to-device memcpy and this library's refresh
    kernel (a bf16 copy) on the same 1 GiB.  GB/s counts bytes read plus
    bytes written, at the median of `reps` launches.  The kernels of the
    path all read and write, so the copy is the ceiling they are compared
    with (frac_of_copy_ceiling)."""
    import torch
    from paper_2407_01614_amd import zpp
    if not os.path.exists(CEILING_LIB):
        raise RuntimeError("%s is not built: run __graft_entry__.build()" % CEILING_LIB)
    lib = ctypes.CDLL(CEILING_LIB)
    for fn in ("zppc_read_stream", "zppc_write_stream", "zppc_copy_stream"):
        getattr(lib, fn).restype = ctypes.c_int
    nbytes = 1 << 30
    src = torch.ones(nbytes // 2, dtype=torch.int16, device="cuda")
    dst = torch.empty_like(src)
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    stream = torch.cuda.current_stream()
    sh = ctypes.c_void_p(zpp.stream_handle(stream))
    vp = lambda t: ctypes.c_void_p(t.data_ptr())

    def check(rc):
        if rc != 0:
            raise RuntimeError("ceiling stream launch failed: hipError %d" % rc)

    streams = (
        ("read_only", nbytes, lambda: check(lib.zppc_read_stream(vp(src), ctypes.c_size_t(nbytes),
                                                                 vp(sink), sh))),
        ("write_only", nbytes, lambda: check(lib.zppc_write_stream(
            vp(dst), ctypes.c_size_t(nbytes), ctypes.c_uint32(0x3F803F80), sh))),
        ("copy", 2 * nbytes, lambda: check(lib.zppc_copy_stream(vp(dst), vp(src),
                                                                ctypes.c_size_t(nbytes), sh))),
        ("hipMemcpyAsync_d2d", 2 * nbytes, lambda: dst.copy_(src)),
        ("refresh_kernel", 2 * nbytes, lambda: zpp.refresh_secondary(dst, src, stream=stream)))
    res = {}
    for name, moved, fn in streams:
        fn()
        evs = []
        for _ in range(reps):
            a, b = zpp.Event(timing=True), zpp.Event(timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            evs.append((a, b))
        torch.cuda.synchronize()
        med = sorted(a.elapsed_ms(b) for a, b in evs)[reps // 2]
        gbps = moved / (med * 1e-3) / 1e9
        res[name] = {"GB/s": round(gbps, 1), "frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4)}
    assert int(sink.item()) == 0
    del src, dst, sink
    res["bytes"] = "1 GiB read and/or 1 GiB written; GB/s = bytes read + bytes written"
    return res


def patterns(wl, reps=20):
    """The access patterns of the Adam step, the dequant-gather and the int8
    quantizer at this workload's sizes (include/zpp_ceiling.h: the same
    loads and stores in the same lane layout, launch shape and residency,
    the arithmetic replaced by an xor), each on buffers of its own, timed
    with events like the ceilings (median of `reps` launches).  A kernel's
    `frac_of_pattern` is its GB/s over its pattern's: 1 or more means its
    arithmetic costs nothing beyond its memory traffic."""
    import torch
    from paper_2407_01614_amd import zpp
    from paper_2407_01614_amd.workloads import BYTES_ADAM, bytes_gather, bytes_quant
    lib = ctypes.CDLL(CEILING_LIB)
    for fn in ("zppc_adam_pattern", "zppc_gather_pattern", "zppc_quant_pattern"):
        getattr(lib, fn).restype = ctypes.c_int
    stream = torch.cuda.current_stream()
    sh = ctypes.c_void_p(zpp.stream_handle(stream))
    vp = lambda t: ctypes.c_void_p(t.data_ptr())

    def check(rc):
        if rc != 0:
            raise RuntimeError("access-pattern launch failed: hipError %d" % rc)

    def timed(fn):
        fn()
        evs = []
        for _ in range(reps):
            a, b = zpp.Event(timing=True), zpp.Event(timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            evs.append((a, b))
        torch.cuda.synchronize()
        return sorted(a.elapsed_ms(b) for a, b in evs)[reps // 2]

    res = {}
    B = wl.block
    # Adam: n rounded down to whole 256-element tiles
    n = wl.n // 256 * 256
    p, m, v, g = (torch.empty(n, dtype=torch.float32, device="cuda") for _ in range(4))
    out = torch.empty(n, dtype=torch.int16, device="cuda")
    ms = timed(lambda: check(lib.zppc_adam_pattern(vp(p), vp(m), vp(v), vp(g), vp(out),
                                                   ctypes.c_size_t(n), sh)))
    res["adam"] = (n, BYTES_ADAM * n, ms)
    del p, m, v, g, out
    # the gather: the layer's N codes (whole 512-element rows) as one array
    N = wl.layer_elems // 512 * 512
    codes = torch.empty(N, dtype=torch.int8, device="cuda")
    scales = torch.ones(N // B, dtype=torch.float32, device="cuda")
    out = torch.empty(N, dtype=torch.int16, device="cuda")
    ms = timed(lambda: check(lib.zppc_gather_pattern(vp(codes), vp(scales), vp(out),
                                                     ctypes.c_size_t(N), sh)))
    res["gather"] = (N, bytes_gather(N, 1, N, B), ms)
    del codes, scales, out
    # the quantizer: n rounded down to whole workgroups of 16 blocks
    nq = wl.n // 4096 * 4096
    src = torch.empty(nq, dtype=torch.int16, device="cuda")
    codes = torch.empty(nq, dtype=torch.int8, device="cuda")
    scales = torch.empty(nq // B, dtype=torch.float32, device="cuda")
    ms = timed(lambda: check(lib.zppc_quant_pattern(vp(src), vp(codes), vp(scales),
                                                    ctypes.c_size_t(nq), sh)))
    res["quant"] = (nq, bytes_quant(nq, B), ms)
    del src, codes, scales
    torch.cuda.empty_cache()
    out = {}
    for k, (elems, nbytes, ms) in res.items():
        gbps = nbytes / (ms * 1e-3) / 1e9
        out[k] = {"elements": elems, "bytes": nbytes, "median_us": round(ms * 1e3, 2),
                  "GB/s": round(gbps, 1), "frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4)}
    return out


def block_sizes(wl, reps=20, blocks=(256, 192, 320, 1088, 4032)):
    """The kernels whose layout depends on the quantization block, at this
    workload's partition and a few blocks other than its own: the int8
    quantizer alone and with the secondary copy, the int4 quantizer and the
    fused step (for blocks outside 64-512 the step with its copies, then the
    quantizer over the primary).  Median of `reps` calls per kernel and
    block, each call timed with events on the current stream (a call of
    the fused step may be two kernels)."""
    import torch
    from paper_2407_01614_amd import synth, zpp
    from paper_2407_01614_amd.workloads import (bytes_fused, bytes_quant, bytes_quant_i4,
                                                bytes_refresh_quant)
    stream = torch.cuda.current_stream()
    n = wl.n

    def timed(fn):
        fn()
        evs = []
        for _ in range(reps):
            a, b = zpp.Event(timing=True), zpp.Event(timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            evs.append((a, b))
        torch.cuda.synchronize()
        return sorted(a.elapsed_ms(b) for a, b in evs)[reps // 2]

    x = synth.device_bf16_weights(n, wl.cfg_id, rank=0)
    sec = torch.empty_like(x)
    codes = torch.empty(n, dtype=torch.int8, device="cuda")
    c4 = torch.empty((n + 1) // 2, dtype=torch.uint8, device="cuda")
    scales = torch.empty(n // 64 + 1, dtype=torch.float32, device="cuda")
    p = synth.device_normal_f32(n, synth.WEIGHT_STD, wl.cfg_id, synth.KIND_MASTER)
    g = synth.device_normal_f32(n, synth.GRAD_STD, wl.cfg_id, synth.KIND_GRAD)
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    prim = torch.empty_like(x)
    hp = dict(wl.adam)
    out = {}
    for B in blocks:
        calls = {
            "quant_i8": (lambda: zpp.quantize_blockwise_i8(x, codes, scales, block=B),
                         bytes_quant(n, B)),
            "refresh_quant_i8": (lambda: zpp.refresh_quantize_i8(sec, x, codes, scales, block=B),
                                 bytes_refresh_quant(n, B)),
            "quant_i4": (lambda: zpp.quantize_blockwise_i4(g, c4, scales, block=B),
                         bytes_quant_i4(n, B)),
            "fused_step_refresh_quant": (
                lambda: zpp.adam_step_refresh_quantize(p, m, v, g, prim, sec, codes, scales,
                                                       step=2, block=B, **hp),
                bytes_fused(n, B)),
        }
        row = {}
        for name, (call, nbytes) in calls.items():
            ms = timed(call)
            gbps = nbytes / (ms * 1e-3) / 1e9
            row[name] = {"bytes": nbytes, "median_us": round(ms * 1e3, 2),
                         "GB/s": round(gbps, 1), "frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4)}
        out[str(B)] = row
    return out


def _chunks(n, parts, align):
    """[a, b) ranges covering [0, n), each boundary a multiple of `align`."""
    step = max(align, -(-n // parts) // align * align)
    return [(a, min(n, a + step)) for a in range(0, n, step)]


def cpu_baseline(wl, frac, threads=1, steps=1):
    """Time the CPU oracle (as it stands) on a `frac` sample of the workload
    for `steps` consecutive steps: Adam on frac*n (all n at frac = 1; step
    t = 1, 2, ..., each from the state the previous one left), refresh and
    quantization of frac*n, gather of a frac*N layer from P' shards.  With threads > 1 each
    op's elements are split into block-aligned ranges, and the same oracle
    calls run on the ranges from a pool of that many threads (the calls
    release the GIL).  Inputs come from the same seeded generators;
    generation is not timed."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor
    import oracle
    from paper_2407_01614_amd import synth
    from paper_2407_01614_amd.workloads import (BYTES_ADAM, BYTES_REFRESH, bytes_gather,
                                                bytes_quant, secondary_elems)
    B = wl.block
    # the whole partition at full size (short last block included), else a
    # whole number of blocks
    n = wl.n if frac >= 1 else max(B, int(wl.n * frac) // B * B)
    N = max(B * wl.secondary_world, int(wl.layer_elems * frac))
    s = secondary_elems(N, wl.secondary_world, B)
    p = synth.master_weights(n, wl.cfg_id)
    g = synth.gradients(n, wl.cfg_id)
    z = np.zeros(n, np.float32)
    w = synth.bf16_weights(wl.secondary_world * s, wl.cfg_id)
    ranges = _chunks(n, threads, B)
    pool = ThreadPoolExecutor(threads) if threads > 1 else None

    def run(fn, items):
        return list(pool.map(fn, items)) if pool else [fn(x) for x in items]

    secs_by = {"adam": 0.0, "refresh": 0.0, "quant": 0.0, "gather": 0.0}
    state = [(p[a:b], z[a:b], z[a:b]) for a, b in ranges]
    quants = [oracle.quantize_blockwise_i8(w[j * s:(j + 1) * s], B)
              for j in range(wl.secondary_world)]
    # shard j holds layer elements [j s, (j+1) s); each piece of a shard is
    # gathered into its own place of the layer
    pieces = [(j, a, b) for j in range(wl.secondary_world)
              for a, b in _chunks(s, max(1, threads // wl.secondary_world), B)
              if j * s + a < N]
    for t in range(1, steps + 1):
        t0 = time.perf_counter()
        res = run(lambda k: oracle.adam_step(*state[k], g[ranges[k][0]:ranges[k][1]], step=t,
                                             **wl.adam), range(len(ranges)))
        t1 = time.perf_counter()
        state = [r[:3] for r in res]
        sec = run(oracle.refresh, [r[3] for r in res])
        t2 = time.perf_counter()
        run(lambda x: oracle.quantize_blockwise_i8(x, B), sec)
        t3 = time.perf_counter()
        run(lambda q: oracle.dequant_gather_layer(
            [quants[q[0]][0][q[1]:q[2]]], [quants[q[0]][1][q[1] // B:-(-q[2] // B)]],
            q[2] - q[1], B, min(q[2] - q[1], N - q[0] * s - q[1])), pieces)
        t4 = time.perf_counter()
        for k, dt in zip(secs_by, (t1 - t0, t2 - t1, t3 - t2, t4 - t3)):
            secs_by[k] += dt
    if pool:
        pool.shutdown()
    secs = sum(secs_by.values())
    nbytes = steps * (BYTES_ADAM * n + BYTES_REFRESH * n + bytes_quant(n, B)
                      + bytes_gather(s, wl.secondary_world, N, B))
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    cpu = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return {"value": round(nbytes / secs / 1e9, 3), "unit": "GB/s", "cores": threads,
            "kind": "oracle", "host_cpu": cpu, "host_logical_cpus": os.cpu_count(),
            "sample": "%s at %.3g of full size, %d step(s): Adam+refresh+quant on %d elements, "
                      "gather of a %d-element layer from %d shards; %d thread(s), %.2f s of "
                      "wall time" % (wl.name, frac, steps, n, N, wl.secondary_world, threads, secs),
            "seconds": {k: round(v, 3) for k, v in secs_by.items()}}


# The oracle at the workloads other than the benchmarked one: (fraction, steps)
# for one thread, then for all host threads, chosen so that each leg takes
# about 0.1-8 s of CPU time (Falcon-40B's all-threads leg runs its 10 steps).
CPU_OTHER_SAMPLES = {
    "tiny": ((1.0, 2), (1.0, 2)),
    "falcon-7b-layer": ((0.5, 2), (1.0, 2)),
    "llama-2-7b": ((0.1, 2), (1.0, 2)),
    "llama-2-13b": ((0.1, 2), (1.0, 2)),
    "falcon-40b": ((0.05, 2), (1.0, 10)),
}


def cpu_baseline_others(skip):
    """The CPU oracle's rate at every other workload: one thread on a bounded
    sample, and all host threads (at most 16) on the whole partition."""
    from paper_2407_01614_amd.workloads import WORKLOADS
    out = {}
    for name, ((f1, k1), (fa, ka)) in CPU_OTHER_SAMPLES.items():
        if name == skip:
            continue
        wl = WORKLOADS[name]
        legs = {}
        for leg, frac, steps, threads in (("one_thread", f1, k1, 1),
                                          ("all_cores", fa, ka, host_threads())):
            r = cpu_baseline(wl, frac, threads, steps=steps)
            legs[leg] = {"value": r["value"], "unit": r["unit"], "cores": r["cores"],
                         "sample": r["sample"]}
        out[name] = legs
    return out


def sustain(pipe, step_bytes, seconds, chunk=50):
    """The headline path (one stream, in order) run back to back for about
    `seconds` of wall time, synchronised every `chunk` steps to read the
    clock: the rate the GPU holds over many seconds, not only over the timed
    steps."""
    import torch
    pipe.fused, pipe.sync, pipe.overlap, pipe.timing, pipe.streams = False, "event", True, None, 1
    torch.cuda.synchronize()
    steps, t0 = 0, time.perf_counter()
    while True:
        for _ in range(chunk):
            pipe.step()
        steps += chunk
        pipe.wait()
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        if el >= seconds:
            break
    gbps = step_bytes * steps / el / 1e9
    return {"seconds": round(el, 2), "steps": steps, "ms_per_step": round(el * 1e3 / steps, 4),
            "GB/s": round(gbps, 1), "frac_of_peak": round(gbps / HBM_PEAK_GBPS, 4)}


def gpu_clock_state():
    """Clock policy of GPU 0 as amd-smi reports it (graphics clock range and
    whether it is locked, HBM clock) and its market name, or None.  Called before this process
    initialises the GPU, so the query runs in a child of a process without a
    GPU context; the current clocks are idle values then, the ranges are what
    the run may use."""
    import subprocess

    def query(*args):
        res = subprocess.run(["amd-smi", *args, "--json"], capture_output=True, text=True,
                             timeout=20)
        return json.loads(res.stdout)["gpu_data"][0]

    try:
        clk = query("metric", "--clock")["clock"]
        gfx, mem = clk["gfx_0"], clk["mem_0"]
        state = {"gfx_mhz_min": gfx["min_clk"]["value"], "gfx_mhz_max": gfx["max_clk"]["value"],
                 "gfx_clock_locked": gfx["clk_locked"], "gfx_deep_sleep": gfx["deep_sleep"],
                 "hbm_mhz": mem["clk"]["value"], "source": "amd-smi metric --clock"}
    except Exception:
        return None
    try:
        state["market_name"] = query("static", "--asic")["asic"]["market_name"]
    except Exception:
        pass
    return state


def host_threads():
    """Threads for the all-cores CPU baseline: the CPUs this process may run
    on, at most 16 (the host share of one GPU)."""
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return max(1, min(16, os.cpu_count() or 1))


def main():
    args = parse()
    if args.gpus != 1:
        print("bench.py measures one GPU only: the partition path is rank-local and the other "
              "ranks' shards are simulated in this GPU's memory; --gpus %d is not supported"
              % args.gpus, file=sys.stderr)
        sys.exit(2)

    clocks = None if args.no_clock_query else gpu_clock_state()
    import torch
    from paper_2407_01614_amd.pipeline import PartitionPipeline
    from paper_2407_01614_amd.workloads import WORKLOADS

    wl = WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    if args.copy_calibration:
        src = torch.ones(1 << 30, dtype=torch.int8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    pipe = PartitionPipeline(wl)
    pipe.load_synthetic()

    def run(fused, sync, timing, overlap=True, streams=1, live=None):
        """W warm-up steps, then K timed steps exactly as the path runs them;
        the kernels named in `live` carry a timing-event pair (events without
        the system-scope fence, which cost the stream next to nothing) in
        those K steps.  With `timing`, K more steps follow with such a pair
        around every kernel on that kernel's own stream (the pipeline then
        runs each kernel alone), for the per-kernel table."""
        pipe.fused, pipe.sync, pipe.overlap, pipe.timing = fused, sync, overlap, None
        pipe.streams = streams
        for _ in range(args.warmup):
            pipe.step()
        pipe.wait()
        torch.cuda.synchronize()
        if live:
            pipe.enable_timing(kernels=live, system_fence=False)
        t0 = time.perf_counter()
        for _ in range(args.steps):
            pipe.step()
        pipe.wait()
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3 / args.steps
        live_times = pipe.kernel_times_ms() if live else None
        pipe.timing = None
        times = None
        if timing:
            pipe.enable_timing(system_fence=False)
            for _ in range(args.steps):
                pipe.step()
            pipe.wait()
            times = pipe.kernel_times_ms()
            pipe.timing = None
        if live:
            return ms, times, pipe.kernel_bytes(), pipe.step_bytes(), live_times
        return ms, times, pipe.kernel_bytes(), pipe.step_bytes()

    # the headline: the path in order on one stream (the stream order is the
    # fix), the Adam launches timed inside its K timed steps; then the same
    # kernels on three streams ordered by events
    ms_per_step, times, kb, step_bytes, live_times = run(False, "event", True, live={"adam"})
    sustained = sustain(pipe, step_bytes, args.sustain_s) if args.sustain_s > 0 else None
    three_ms = run(False, "event", False, overlap=True, streams=3)[0]
    fused_ms, fused_times, fused_kb, fused_step_bytes = run(True, "event", True)
    # the refresh and its quantization as one pass (zpp_refresh_quantize_i8)
    pipe.fuse_copy = True
    fc_ms, fc_times, fc_kb, fc_step_bytes = run(False, "event", True)
    pipe.fuse_copy = False
    sync_ab = {}
    for mode in ("event", "host", "none"):
        sync_ab[mode] = round(run(False, mode, False, overlap=False, streams=3)[0], 4)
    ceil = ceilings()
    copy_gbps = ceil["copy"]["GB/s"]
    pats = patterns(wl) if wl.block == 256 else None
    torch_ctx = torch_adamw_context(wl, args.steps)
    # the whole iteration seen by the rank with qgZ: the int4 quantization of
    # its gradient into its send buffer (the send), the receive of 8 int4
    # copies of its partition's gradient delivered into one interleaved
    # receive buffer (their mean) feeding the step, as its own kernel, fused
    # into the partition step, and inside the single pass of step, refresh
    # and quantization
    from paper_2407_01614_amd import synth as _synth
    from paper_2407_01614_amd.pipeline import GradientExchange
    pipe.exchange = GradientExchange(wl.n, 8, wl.block, interleaved=True)
    for q in range(8):
        g = _synth.device_normal_f32(wl.n, _synth.GRAD_STD, wl.cfg_id, _synth.KIND_GRAD, rank=q)
        pipe.exchange.quantize(q, g)
        del g
    pipe.send_grad = _synth.device_normal_f32(wl.n, _synth.GRAD_STD, wl.cfg_id,
                                              _synth.KIND_GRAD, rank=8)
    torch.cuda.synchronize()
    pipe.fuse_receive = False
    ilr_ms, ilr_times, ilr_kb, ilr_step_bytes = run(False, "event", True)
    ilr_gbps = ilr_step_bytes / (ilr_ms * 1e-3) / 1e9
    pipe.fuse_receive = True
    il_ms, il_times, il_kb, il_step_bytes = run(False, "event", True)
    il_gbps = il_step_bytes / (il_ms * 1e-3) / 1e9
    ilf_ms, ilf_times, ilf_kb, ilf_step_bytes = run(True, "event", True)
    ilf_gbps = ilf_step_bytes / (ilf_ms * 1e-3) / 1e9
    pipe.fuse_receive = False
    pipe.exchange = None
    pipe.send_grad = None
    qgz_kernels = kernel_table(ilr_kb, ilr_times, copy_gbps)
    qgz = {"sources": 8, "from": "step_with_qgz_receive (timed inside its steps)",
           "quant_i4": qgz_kernels["quant_i4"],
           "dequant_reduce_i4_interleaved": qgz_kernels["reduce_i4"]}
    value = step_bytes / (ms_per_step * 1e-3) / 1e9
    kernels = kernel_table(kb, times, copy_gbps)
    for k in ("adam", "gather", "quant"):
        if pats and k in kernels:
            kernels[k]["frac_of_pattern"] = round(kernels[k]["GB/s"] / pats[k]["GB/s"], 4)
    fused_kernels = kernel_table(fused_kb, fused_times, copy_gbps)
    fused_gbps = fused_step_bytes / (fused_ms * 1e-3) / 1e9
    sr_us = kernels["adam"]["mean_us"] + kernels["refresh"]["mean_us"]
    sr_gbps = (kb["adam"] + kb["refresh"]) / (sr_us * 1e-6) / 1e9

    traffic = measured_traffic(args.traffic, wl.name, "adam", TRAFFIC_SOURCES["adam"])

    # the dominant kernel's mean launch duration over the K timed steps
    adam_live = live_times["adam"]
    adam_mean_s = sum(adam_live) / len(adam_live) * 1e-3
    achieved = kb["adam"] / adam_mean_s / 1e9
    line = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "ms_per_step_three_streams": {"overlap": round(three_ms, 4),
                                      "without_overlap": sync_ab["event"]},
        "sustained": sustained,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": "%s rank shard: n=%d fp32 master/m/v/grad, bf16 primary and "
                               "secondary, int8 blocks of %d; %s of a %d-element layer "
                               "from %d secondary shards of %d"
                               % (wl.name, wl.n, wl.block,
                                  "gather" if wl.layers_gathered == 1 else
                                  "%d gathers (over %d stored layers)"
                                  % (wl.layers_gathered, wl.distinct_layers),
                                  wl.layer_elems, wl.secondary_world, wl.shard_elems),
                   "n": wl.n, "layer_elems": wl.layer_elems, "secondary_world": wl.secondary_world,
                   "shard_elems": wl.shard_elems, "block": wl.block,
                   "layers_gathered_per_step": wl.layers_gathered},
        "roofline": {"bound": "hbm", "kernel": "adam_partition_step",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": round(achieved / HBM_PEAK_GBPS, 4), "traffic": traffic,
                     "mean_launch_us": round(adam_mean_s * 1e6, 2),
                     "launches": len(adam_live)},
        "step_refresh": {"GB/s": round(sr_gbps, 1), "frac_of_peak": round(sr_gbps / HBM_PEAK_GBPS, 4)},
        "gather": {"GB/s": kernels["gather"]["GB/s"],
                   "frac_of_peak": kernels["gather"]["frac_of_peak"]},
        "kernels": kernels,
        "fused_step_refresh_quant": {
            "ms_per_step": round(fused_ms, 4), "GB/s": round(fused_gbps, 1),
            "frac_of_peak": round(fused_gbps / HBM_PEAK_GBPS, 4), "kernels": fused_kernels},
        "step_with_fused_refresh_quant": {
            "ms_per_step": round(fc_ms, 4),
            "GB/s": round(fc_step_bytes / (fc_ms * 1e-3) / 1e9, 1),
            "frac_of_peak": round(fc_step_bytes / (fc_ms * 1e-3) / 1e9 / HBM_PEAK_GBPS, 4),
            "kernels": kernel_table(fc_kb, fc_times, copy_gbps)},
        "sync_ab_ms_per_step": sync_ab,
        "ceilings": ceil,
        "access_patterns": pats,
        "torch_fused_adamw_context": dict(
            torch_ctx, speedup_of_partition_step=round(
                torch_ctx["ms_per_step"] / (kernels["adam"]["mean_us"] * 1e-3), 3)),
        "qgz_gradient_side": qgz,
        "step_with_qgz_receive": {
            "ms_per_step": round(ilr_ms, 4), "GB/s": round(ilr_gbps, 1),
            "frac_of_peak": round(ilr_gbps / HBM_PEAK_GBPS, 4),
            "kernels": kernel_table(ilr_kb, ilr_times, copy_gbps)},
        "step_with_fused_qgz_receive": {
            "ms_per_step": round(il_ms, 4), "GB/s": round(il_gbps, 1),
            "frac_of_peak": round(il_gbps / HBM_PEAK_GBPS, 4),
            "kernels": kernel_table(il_kb, il_times, copy_gbps)},
        "step_with_qgz_receive_single_pass": {
            "ms_per_step": round(ilf_ms, 4), "GB/s": round(ilf_gbps, 1),
            "frac_of_peak": round(ilf_gbps / HBM_PEAK_GBPS, 4),
            "kernels": kernel_table(ilf_kb, ilf_times, copy_gbps)},
        "device": torch.cuda.get_device_properties(0).gcnArchName,
        "gpu": {"name": torch.cuda.get_device_name(0),
                "compute_units": torch.cuda.get_device_properties(0).multi_processor_count,
                "memory_gib": round(torch.cuda.get_device_properties(0).total_memory / 2**30, 1),
                "clocks": clocks},
    }
    del pipe
    torch.cuda.empty_cache()
    line["forward_gather_qwz"] = forward_gather_measure(wl, args.steps)
    torch.cuda.empty_cache()
    line["block_sizes"] = block_sizes(wl)
    torch.cuda.empty_cache()
    if args.cpu_sample > 0:
        line["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample, steps=args.cpu_steps)
        line["cpu_baseline_all_cores"] = cpu_baseline(wl, args.cpu_sample, host_threads(),
                                                      steps=args.cpu_steps)
        if args.cpu_other:
            line["cpu_baseline_other_workloads"] = cpu_baseline_others(wl.name)
    else:
        line["cpu_baseline"] = None
        line["cpu_baseline_all_cores"] = None
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
