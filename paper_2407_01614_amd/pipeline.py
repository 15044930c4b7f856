"""One simulated rank's partition path, on three HIP streams or on one.

Per iteration (Algorithm 1 seen from one rank, one GPU):
  compute stream : optimizer step on the rank's partition -> bf16 primary
  copy stream    : refresh the hpZ secondary copy from the primary, then
                   quantize it (qwZ)
  comm stream    : backward gather of one layer from the P' node-local
                   secondary shards, dequantizing on the way

With `streams=1` the same kernels run in that order on the compute stream
alone: the order of the stream is then the fix (the gather cannot start
before the quantization of the copy it reads has finished) and no event is
needed.  On one GPU this is the faster arrangement, because every kernel is
bound by HBM bandwidth, so overlapping two of them gains nothing, while each
edge between streams costs the device some microseconds.  The three-stream
form is the one a training step uses when the copy overlaps the forward
pass's compute.

Local rank 0's shard of the gathered layer is s codes of this rank's own
freshly quantized secondary; the other P' - 1 shards stand for the peers of
the secondary group and live in this GPU's memory.  A step gathers
`wl.layers_gathered` layers (the backward pass visits every layer once),
cycling over `wl.distinct_layers` stored layers: layer k takes the local
codes [k s, (k+1) s) and its own set of peer shards.  The gathers wait on the
quantize's event (the ordering fix); across iterations the write-after-read
edges on the primary and the codes are events too, so one iteration's gathers
overlap the next iteration's optimizer step.

Buffers are laid out flat in HBM, one allocation per array, 256-byte
aligned (torch's allocator), so every kernel takes its 16-byte vector path.
"""
import functools

import numpy as np
import torch

from . import synth
from . import zpp
from .workloads import (BYTES_ADAM, BYTES_REFRESH, bytes_fused, bytes_fused_receive,
                        bytes_gather, bytes_quant, bytes_quant_i4, bytes_receive_adam,
                        bytes_reduce_i4, bytes_refresh_quant)


SYNC_MODES = ("event", "host", "none")


class PartitionPipeline:
    """`fused`: one pass for step + refresh + quantize instead of three
    kernels.  `sync`: how the gather is ordered after the quantization on
    three streams -- "event" (the paper's fix, as a device-side stream wait),
    "host" (the host blocks on the event before it enqueues the gather: the
    fix as a host-side wait) or "none" (stock hpZ: no edge at all; the gather
    may read codes that are not written yet, so only its timing means
    anything).  `streams=1` runs every kernel on the compute stream in path
    order; `sync` and `overlap` do not apply there.  `qgz_sources` > 0 opens
    every step with the qgZ receive of that many int4 gradient copies, as its
    own dequantize-and-reduce kernel writing `grad`, or, with `fuse_receive`,
    inside the partition step (`zpp_qgz_receive_adam_step`, no `grad`
    written), and with `fused` too, inside the single pass of step, refresh
    and quantization (`zpp_qgz_receive_step_refresh_quantize`).
    `qgz_interleaved` keeps the int4 copies in one interleaved receive buffer
    (`GradientExchange`), read by the `..._interleaved` entry points.  With
    an exchange, setting `send_grad` (an fp32 tensor of n: one partition's
    worth of this rank's gradient, from the backward pass) opens every step
    with its int4 quantization into the exchange's send buffer (plain
    layout), the sender's share of the exchange; the receive slots stand for
    the copies the exchange delivers from the ranks.  `fuse_copy` runs the
    refresh and the quantization of the separate-kernel path as one pass
    (`zpp_refresh_quantize_i8`)."""

    def __init__(self, wl, device="cuda", fused=False, sync="event", overlap=True,
                 qgz_sources=0, streams=3, fuse_receive=False, qgz_interleaved=False,
                 fuse_copy=False):
        if sync not in SYNC_MODES:
            raise ValueError("sync must be one of %s" % (SYNC_MODES,))
        if streams not in (1, 3):
            raise ValueError("streams must be 1 or 3")
        self.wl = wl
        self.dev = device
        self.fused = fused
        self.sync = sync
        self.overlap = overlap
        self.streams = streams
        self.fuse_receive = fuse_receive
        self.fuse_copy = fuse_copy
        # with qgz_sources > 0 every step starts with the qgZ receive: the mean
        # of that many int4 copies of this partition's gradient becomes `grad`
        self.exchange = (GradientExchange(wl.n, qgz_sources, wl.block, device,
                                          interleaved=qgz_interleaved)
                         if qgz_sources else None)
        n, s, B = wl.n, wl.shard_elems, wl.block
        K = wl.distinct_layers
        if K < 1 or wl.layers_gathered < 1:
            raise ValueError("a step gathers at least one layer, from at least one stored layer")
        if K * s > n:
            raise ValueError("the local gather shards (%d x %d) must fit in the rank partition (%d)"
                             % (K, s, n))
        f32 = dict(dtype=torch.float32, device=device)
        self.master = torch.empty(n, **f32)
        self.exp_avg = torch.zeros(n, **f32)
        self.exp_avg_sq = torch.zeros(n, **f32)
        self.grad = torch.empty(n, **f32)
        self.primary = torch.empty(n, dtype=torch.int16, device=device)
        self.secondary = torch.empty(n, dtype=torch.int16, device=device)
        self.codes = torch.empty(n, dtype=torch.int8, device=device)
        self.scales = torch.empty((n + B - 1) // B, **f32)
        P2 = wl.secondary_world
        # layer_peers[k] = (codes, scales) of the P' - 1 peer shards of stored layer k
        self.layer_peers = [
            ([torch.empty(s, dtype=torch.int8, device=device) for _ in range(P2 - 1)],
             [torch.empty(s // B, **f32) for _ in range(P2 - 1)]) for _ in range(K)]
        self.peer_codes, self.peer_scales = self.layer_peers[0]
        self.out = torch.empty(wl.layer_elems, dtype=torch.int16, device=device)
        self.compute = torch.cuda.Stream(device)
        self.copy = torch.cuda.Stream(device)
        self.comm = torch.cuda.Stream(device)
        self.ev_primary = zpp.Event()
        self.ev_refresh = zpp.Event()
        self.ev_quant = zpp.Event()
        self.ev_gather = zpp.Event()
        self.send_grad = None
        self.step_count = 0
        self.timing = None
        self._timing_fence = True
        self._prev_streams = streams

    # ------------------------------------------------------------------
    # inputs
    # ------------------------------------------------------------------
    def load(self, master, grad, peer_codes=None, peer_scales=None):
        """Copy host arrays in: the fp32 master shard and its gradient; the
        peers' quantized shards of stored layer 0 if given (else see
        `quantize_peers` and `load_layer_peers`)."""
        self.master.copy_(torch.from_numpy(master))
        self.grad.copy_(torch.from_numpy(grad))
        self.exp_avg.zero_()
        self.exp_avg_sq.zero_()
        if peer_codes is not None:
            self.load_layer_peers(0, peer_codes, peer_scales)
        self.step_count = 0
        torch.cuda.synchronize(self.dev)

    def load_layer_peers(self, k, peer_codes, peer_scales):
        """Copy host arrays in: the P' - 1 peers' codes and scales of stored
        layer k."""
        codes, scales = self.layer_peers[k]
        if len(peer_codes) != len(codes) or len(peer_scales) != len(scales):
            raise ValueError("one codes and one scales array per peer (%d)" % len(codes))
        for t, a in zip(codes, peer_codes):
            t.copy_(torch.from_numpy(a))
        for t, a in zip(scales, peer_scales):
            t.copy_(torch.from_numpy(a))
        torch.cuda.synchronize(self.dev)

    def quantize_peers(self, cfg):
        """Fill the peer shards of every stored layer by quantizing synthetic
        bf16 weights with the library's own quantizer (set-up work, not part
        of a step)."""
        s = self.wl.shard_elems
        for k, (codes, scales) in enumerate(self.layer_peers):
            for j, (c, sc) in enumerate(zip(codes, scales)):
                w = synth.device_bf16_weights(s, cfg, rank=j + 1, it=k, device=self.dev)
                zpp.quantize_blockwise_i8(w, c, sc, block=self.wl.block)
                torch.cuda.synchronize(self.dev)
                del w

    def layer_shards(self, k):
        """Codes and scales of the P' shards of stored layer k, local rank 0
        first: this rank's quantized secondary [k s, (k+1) s), then the peers."""
        s, B = self.wl.shard_elems, self.wl.block
        codes, scales = self.layer_peers[k]
        return ([self.codes[k * s:(k + 1) * s]] + codes,
                [self.scales[k * s // B:(k + 1) * s // B]] + scales)

    def _gathers(self, stream, waits=(), done_after=None):
        """The backward pass's gathers of one step, in layer order on `stream`;
        the first waits on `waits`, the last records `done_after`."""
        wl = self.wl
        G = wl.layers_gathered
        for i in range(G):
            codes, scales = self.layer_shards(i % wl.distinct_layers)
            self._timed("gather", stream, functools.partial(
                zpp.dequant_gather_layer, codes, scales, wl.shard_elems, wl.layer_elems,
                self.out, block=wl.block, stream=stream, wait_events=waits if i == 0 else (),
                done_after=done_after if i == G - 1 else None))

    def load_synthetic(self):
        """Seeded synthetic state drawn on the device: master ~ N(0, 0.02),
        grad ~ N(0, 1e-3), zero moments, peers quantized from N(0, 0.02)."""
        wl = self.wl
        self.master.copy_(synth.device_normal_f32(wl.n, synth.WEIGHT_STD, wl.cfg_id,
                                                  synth.KIND_MASTER, device=self.dev))
        self.grad.copy_(synth.device_normal_f32(wl.n, synth.GRAD_STD, wl.cfg_id, synth.KIND_GRAD,
                                                device=self.dev))
        self.exp_avg.zero_()
        self.exp_avg_sq.zero_()
        self.step_count = 0
        torch.cuda.synchronize(self.dev)
        self.quantize_peers(wl.cfg_id)

    # ------------------------------------------------------------------
    # one iteration
    # ------------------------------------------------------------------
    def enable_timing(self, kernels=None, system_fence=True):
        """Record a HIP timing-event pair around every kernel (or those named
        in `kernels`), on the stream that kernel runs on.  With
        `system_fence=False` the events skip the system-scope fence, so that
        timing one kernel inside an otherwise uninstrumented run costs the
        stream next to nothing."""
        self.timing = {k: [] for k in self.kernel_bytes() if kernels is None or k in kernels}
        self._timing_fence = system_fence

    def _timed(self, name, stream, fn):
        if self.timing is None or name not in self.timing:
            fn()
            return
        a = zpp.Event(timing=True, system_fence=self._timing_fence)
        b = zpp.Event(timing=True, system_fence=self._timing_fence)
        a.record(stream)
        fn()
        b.record(stream)
        self.timing[name].append((a, b))

    def step(self):
        """Enqueue one iteration.  Edges: the step reads the gradient and
        writes the primary; the refresh reads the primary (after the step) and
        writes the secondary; the quantization reads the secondary and writes
        codes and scales; the gathers read the codes (after the quantization:
        the fix) and write the layers.  Across iterations only the
        write-after-read edges are needed: the next step waits for this
        refresh (the primary), the next quantization for this step's last
        gather (the codes), so the gathers of one iteration may overlap the
        next step.
        With `overlap` off, or while timing kernels, the next step waits for
        the whole iteration instead, so each kernel runs alone."""
        wl = self.wl
        n, B = wl.n, wl.block
        self.step_count += 1
        t = self.step_count
        if self.streams == 1:
            self._step_one_stream(t)
            self._prev_streams = 1
            return
        self._prev_streams = 3
        serial = not self.overlap or self.timing is not None
        if t > 1:
            if serial or self.fused:
                # the fused kernel writes the codes, which the last gather reads
                zpp.stream_wait(self.compute, self.ev_gather)
            else:
                # the last refresh has read the primary
                zpp.stream_wait(self.compute,
                                self.ev_quant if self.fuse_copy else self.ev_refresh)
        self._send(self.compute)
        if self._receive_apart():
            self._timed("reduce_i4", self.compute,
                        lambda: self.exchange.reduce(self.grad, stream=self.compute))
        if self.fused:
            self._fused_pass(t, self.compute, self.ev_quant)
        else:
            self._partition_step(t, self.compute)
            self.ev_primary.record(self.compute)
            if self.timing is not None:
                # the refresh waits on the primary itself (wait_before); a
                # timed run waits first, so that the start of the timing pair
                # follows the wait
                zpp.stream_wait(self.copy, self.ev_primary)
            if self.fuse_copy:
                self._copy_and_quantize(t, serial)
            else:
                self._copy_then_quantize(t, serial)
        waits = []
        if self.sync == "event":
            # the gather waits on the quantization itself (the fix, through
            # wait_events); a timed run waits first, as for the refresh
            if self.timing is not None:
                zpp.stream_wait(self.comm, self.ev_quant)
            waits = [self.ev_quant]
        elif self.sync == "host":
            self.ev_quant.synchronize()
        self._gathers(self.comm, waits, self.ev_gather)

    def _copy_and_quantize(self, t, serial):
        """Three streams: the refresh and the quantization as one pass on the
        copy stream, after the primary and (across iterations) after the last
        gather read the codes."""
        n, B = self.wl.n, self.wl.block
        if t > 1 and not serial:
            zpp.stream_wait(self.copy, self.ev_gather)
        self._timed("refresh_quant", self.copy, lambda: zpp.refresh_quantize_i8(
            self.secondary, self.primary, self.codes, self.scales, block=B, n=n,
            stream=self.copy, wait_before=self.ev_primary, done_after=self.ev_quant))

    def _copy_then_quantize(self, t, serial):
        """Three streams: the refresh, then the quantization, on the copy
        stream."""
        n, B = self.wl.n, self.wl.block
        self._timed("refresh", self.copy, lambda: zpp.refresh_secondary(
            self.secondary, self.primary, n, stream=self.copy, wait_before=self.ev_primary,
            done_after=self.ev_refresh))
        if t > 1 and not serial:
            # the quantization rewrites the codes the last gather read; in
            # serial order the step already waited for that gather before the
            # partition step, which the copy stream follows
            zpp.stream_wait(self.copy, self.ev_gather)
        self._timed("quant", self.copy, lambda: zpp.quantize_blockwise_i8(
            self.secondary, self.codes, self.scales, block=B, n=n, stream=self.copy,
            done_after=self.ev_quant))

    def _step_one_stream(self, t):
        """The iteration in path order on the compute stream: each kernel
        starts after the one before it, so the refresh reads the finished
        primary and the gather reads finished codes, and the next iteration's
        writes come after this one's reads.  No event is recorded: on one
        stream a record costs the device about 4 us and a wait on it about
        8 us, for an order the stream already gives.  A following
        three-stream iteration stays ordered after this one, since its own
        edges start from the compute stream."""
        wl = self.wl
        n, B = wl.n, wl.block
        cs = self.compute
        if t > 1 and self._prev_streams == 3:
            # the last iteration ran on three streams: join its copy and comm
            # work (the quantization, then the gather) into this stream
            zpp.stream_wait(cs, self.ev_quant)
            zpp.stream_wait(cs, self.ev_gather)
        self._send(cs)
        if self._receive_apart():
            self._timed("reduce_i4", cs, lambda: self.exchange.reduce(self.grad, stream=cs))
        if self.fused:
            self._fused_pass(t, cs, None)
        else:
            self._partition_step(t, cs)
            if self.fuse_copy:
                self._timed("refresh_quant", cs, lambda: zpp.refresh_quantize_i8(
                    self.secondary, self.primary, self.codes, self.scales, block=B, n=n,
                    stream=cs))
            else:
                self._timed("refresh", cs, lambda: zpp.refresh_secondary(
                    self.secondary, self.primary, n, stream=cs))
                self._timed("quant", cs, lambda: zpp.quantize_blockwise_i8(
                    self.secondary, self.codes, self.scales, block=B, n=n, stream=cs))
        self._gathers(cs)

    def _sends(self):
        return self.exchange is not None and self.send_grad is not None

    def _send(self, stream):
        """The qgZ send: the int4 quantization of this rank's gradient into
        the exchange's send buffer, ahead of the receive on the same stream."""
        if self._sends():
            self._timed("quant_i4", stream, lambda: self.exchange.send(
                self.send_grad, stream=stream))

    def _receive_fused(self):
        return self.exchange is not None and self.fuse_receive

    def _receive_apart(self):
        return self.exchange is not None and not self._receive_fused()

    def _fused_pass(self, t, stream, done_after):
        """Step, refresh and quantization in one pass: from `grad`, or with
        the qgZ receive fused in, from the int4 copies of the gradient."""
        wl, B = self.wl, self.wl.block
        if self._receive_fused():
            ex = self.exchange
            if ex.interleaved:
                call = functools.partial(zpp.qgz_receive_step_refresh_quantize_interleaved,
                                         self.master, self.exp_avg, self.exp_avg_sq, ex.codes,
                                         ex.scales, ex.num_src)
            else:
                call = functools.partial(zpp.qgz_receive_step_refresh_quantize, self.master,
                                         self.exp_avg, self.exp_avg_sq, ex.codes, ex.scales)
            self._timed("fused_receive", stream, lambda: call(
                self.primary, self.secondary, self.codes, self.scales, step=t,
                grad_block=ex.block, block=B, scale_out=1.0 / ex.num_src, stream=stream,
                done_after=done_after, **wl.adam))
        else:
            self._timed("fused", stream, lambda: zpp.adam_step_refresh_quantize(
                self.master, self.exp_avg, self.exp_avg_sq, self.grad, self.primary,
                self.secondary, self.codes, self.scales, step=t, block=B, stream=stream,
                done_after=done_after, **wl.adam))

    def _partition_step(self, t, stream):
        """The Adam step of the separate-kernel path: from `grad`, or with the
        qgZ receive fused in, from the int4 copies of the gradient."""
        wl = self.wl
        if self._receive_fused():
            ex = self.exchange
            if ex.interleaved:
                call = functools.partial(zpp.qgz_receive_adam_step_interleaved, self.master,
                                         self.exp_avg, self.exp_avg_sq, ex.codes, ex.scales,
                                         ex.num_src)
            else:
                call = functools.partial(zpp.qgz_receive_adam_step, self.master, self.exp_avg,
                                         self.exp_avg_sq, ex.codes, ex.scales)
            self._timed("receive_adam", stream, lambda: call(
                self.primary, step=t, block=ex.block, scale_out=1.0 / ex.num_src,
                stream=stream, **wl.adam))
        else:
            self._timed("adam", stream, lambda: zpp.adam_partition_step(
                self.master, self.exp_avg, self.exp_avg_sq, self.grad, self.primary, step=t,
                stream=stream, **wl.adam))

    def wait(self):
        """Block the host until every stream of the pipeline is idle."""
        torch.cuda.synchronize(self.dev)

    # ------------------------------------------------------------------
    # accounting
    # ------------------------------------------------------------------
    def launches_per_step(self):
        """How many times each kernel runs in one step."""
        return {k: (self.wl.layers_gathered if k == "gather" else 1) for k in self.kernel_bytes()}

    def step_bytes(self):
        """Algorithmic HBM bytes of one whole step."""
        per = self.launches_per_step()
        return sum(b * per[k] for k, b in self.kernel_bytes().items())

    def kernel_bytes(self):
        """Algorithmic HBM bytes of one launch of each kernel of the step."""
        wl = self.wl
        gather = float(bytes_gather(wl.shard_elems, wl.secondary_world, wl.layer_elems, wl.block))
        out = {}
        if self._sends():
            out["quant_i4"] = float(bytes_quant_i4(wl.n, self.exchange.block))
        if self._receive_apart():
            out["reduce_i4"] = float(bytes_reduce_i4(wl.n, self.exchange.num_src, wl.block))
        if self.fused and self._receive_fused():
            out.update({"fused_receive": float(bytes_fused_receive(
                wl.n, self.exchange.num_src, wl.block, self.exchange.block)), "gather": gather})
            return out
        if self.fused:
            out.update({"fused": float(bytes_fused(wl.n, wl.block)), "gather": gather})
            return out
        if self._receive_fused():
            out["receive_adam"] = float(bytes_receive_adam(wl.n, self.exchange.num_src, wl.block))
        else:
            out["adam"] = BYTES_ADAM * wl.n
        if self.fuse_copy:
            out["refresh_quant"] = float(bytes_refresh_quant(wl.n, wl.block))
        else:
            out.update({"refresh": BYTES_REFRESH * wl.n,
                        "quant": float(bytes_quant(wl.n, wl.block))})
        out["gather"] = gather
        return out

    def kernel_times_ms(self):
        """Per-kernel list of event-measured durations (ms); call after wait()."""
        return {k: [a.elapsed_ms(b) for a, b in v] for k, v in self.timing.items()}


class GradientExchange:
    """The qgZ gradient side of one rank's partition, on one GPU: each of the
    `num_src` sending ranks quantizes its gradient of this rank's partition to
    int4 (sources other than this rank are simulated in this GPU's memory),
    and the rank reduces the copies into the fp32 mean gradient that the
    partition step reads.  With `interleaved` the copies arrive in one
    receive buffer, block by block (the layout of include/zpp.h).  `send`
    quantizes this rank's own gradient into a send buffer of the plain
    layout (`send_codes`, `send_scales`), what a sender hands the exchange."""

    def __init__(self, n, num_src, block=256, device="cuda", interleaved=False):
        self.n, self.num_src, self.block = n, num_src, block
        self.interleaved = interleaved
        nb = (n + block - 1) // block
        if interleaved:
            nc, ns = zpp.interleaved_sizes(n, block, num_src)
            self.codes = torch.zeros(nc, dtype=torch.uint8, device=device)
            self.scales = torch.zeros(ns, dtype=torch.float32, device=device)
        else:
            self.codes = [torch.empty((n + 1) // 2, dtype=torch.uint8, device=device)
                          for _ in range(num_src)]
            self.scales = [torch.empty(nb, dtype=torch.float32, device=device)
                           for _ in range(num_src)]

    def send(self, grad, stream=None, done_after=None):
        if getattr(self, "send_codes", None) is None:
            dev = grad.device
            self.send_codes = torch.empty((self.n + 1) // 2, dtype=torch.uint8, device=dev)
            self.send_scales = torch.empty((self.n + self.block - 1) // self.block,
                                           dtype=torch.float32, device=dev)
        zpp.quantize_blockwise_i4(grad, self.send_codes, self.send_scales, block=self.block,
                                  n=self.n, stream=stream, done_after=done_after)

    def quantize(self, q, grad, stream=None, done_after=None):
        if self.interleaved:
            zpp.quantize_blockwise_i4_interleaved(grad, self.codes, self.scales, source=q,
                                                  num_src=self.num_src, block=self.block,
                                                  n=self.n, stream=stream, done_after=done_after)
        else:
            zpp.quantize_blockwise_i4(grad, self.codes[q], self.scales[q], block=self.block,
                                      n=self.n, stream=stream, done_after=done_after)

    def reduce(self, out, stream=None, wait_events=(), done_after=None):
        if self.interleaved:
            zpp.dequant_reduce_i4_interleaved(self.codes, self.scales, self.num_src, self.n, out,
                                              block=self.block, scale_out=1.0 / self.num_src,
                                              stream=stream, wait_events=wait_events,
                                              done_after=done_after)
            return
        zpp.dequant_reduce_i4(self.codes, self.scales, self.n, out, block=self.block,
                              scale_out=1.0 / self.num_src, stream=stream,
                              wait_events=wait_events, done_after=done_after)
