"""The whole partition path on streams, and the ordering fix of the paper.

Stream layout (one simulated rank, as in the benchmark):
  compute stream : Adam partition step  -> event `primary_ready`
  copy stream    : wait primary_ready, refresh secondary, quantize -> `quant_done`
  comm stream    : wait quant_done (the fix), dequant-gather -> `gather_done`
The next iteration's refresh waits on `gather_done` (the buffer it overwrites
is still being read until then).
"""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from paper_2407_01614_amd import synth
from paper_2407_01614_amd.workloads import WORKLOADS
from parity import (MomentTolerance, assert_adam_close, assert_bits_equal, empty_dev, to_dev,
                    to_host)

pytestmark = pytest.mark.gpu

TINY = WORKLOADS["tiny"]
# The small workload's 1,048,576 elements are read as one rank's partition
# (4 ranks, a 4,194,304-element layer, shards of 2,097,152); the other reading
# takes them as the whole layer (partitions of 262,144, shards of 524,288).
# Both divide evenly; both run.
TINY_READINGS = {
    "rank-partition": TINY,
    "whole-layer": dataclasses.replace(TINY, name="tiny-whole-layer", n=TINY.n // TINY.world,
                                       layer_elems=TINY.n),
}


@pytest.fixture(scope="module")
def zpp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2407_01614_amd import zpp as mod
    return mod


def f32hp(hp):
    return {k: float(np.float32(v)) for k, v in hp.items()}


def oracle_tiny_pipeline(hp, wl=TINY):
    """The small workload on the oracle: 4 ranks step their partitions, the
    forward-gathered layer is their concatenation, local rank j of the
    secondary group (P' = 2) copies its slice, quantizes it, and the backward
    gather rebuilds the layer."""
    n, P, P2, B = wl.n, wl.world, wl.secondary_world, wl.block
    N = wl.layer_elems
    ranks = []
    layer = np.empty(N, np.uint16)
    for r in range(P):
        p = synth.master_weights(n, wl.cfg_id, r)
        g = synth.gradients(n, wl.cfg_id, r)
        z = np.zeros(n, np.float32)
        res = oracle.adam_step(p, z, z, g, step=1, **hp)
        ranks.append(res)
        b, e = oracle.primary_slice(N, P, r)
        layer[b:e] = res[3]
    s = oracle.secondary_shard_elems(N, P2, B)
    secondaries = []
    quants = []
    for j in range(P2):
        b, e = oracle.secondary_slice(N, P2, j, B)
        sec = np.zeros(s, np.uint16)
        sec[:e - b] = oracle.refresh(layer[b:e])
        secondaries.append(sec)
        quants.append(oracle.quantize_blockwise_i8(sec, B))
    out = oracle.dequant_gather_layer([q[0] for q in quants], [q[1] for q in quants], s, B, N)
    return ranks, layer, secondaries, quants, out


def assert_downstream(g_prim, r_prim, g_codes, g_scales, r_codes, r_scales, B, what):
    """Quantized results computed from the GPU's and the oracle's own primary:
    bit-exact in every block whose inputs agree (the primaries may differ by 1
    bf16 ulp at a few elements); elsewhere codes move by at most 1."""
    same = (g_prim.reshape(-1, B) == r_prim.reshape(-1, B)).all(axis=1)
    assert same.mean() > 0.99, what
    gc, rc = g_codes.reshape(-1, B), r_codes.reshape(-1, B)
    assert_bits_equal(gc[same], rc[same], what + " codes")
    assert_bits_equal(g_scales[same], r_scales[same], what + " scales")
    assert np.abs(gc[~same].astype(int) - rc[~same]).max(initial=0) <= 1
    return same


@pytest.mark.parametrize("reading", sorted(TINY_READINGS))
def test_tiny_pipeline_on_streams(zpp, reading):
    wl = TINY_READINGS[reading]
    hp = f32hp(wl.adam)
    n, P, P2, B, N = wl.n, wl.world, wl.secondary_world, wl.block, wl.layer_elems
    s = wl.shard_elems
    assert P * n == N and P2 * s == N
    compute, copy, comm = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    layer = empty_dev(N, np.uint16, fill=0x7FC0)
    states, grads = [], []
    for r in range(P):
        states.append((to_dev(synth.master_weights(n, wl.cfg_id, r)),
                       torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")))
        grads.append(to_dev(synth.gradients(n, wl.cfg_id, r)))
    torch.cuda.synchronize()
    primary_ready = zpp.Event()
    for r in range(P):
        p, m, v = states[r]
        zpp.adam_partition_step(p, m, v, grads[r], layer[r * n:(r + 1) * n], step=1,
                                stream=compute, **hp)
    primary_ready.record(compute)
    secs = [empty_dev(s, np.uint16, fill=0x7FC0) for _ in range(P2)]
    codes = [empty_dev(s, np.int8, fill=0) for _ in range(P2)]
    scales = [empty_dev(s // B, np.float32, fill=float("nan")) for _ in range(P2)]
    quant_done = [zpp.Event() for _ in range(P2)]
    gather_done = zpp.Event()
    for j in range(P2):
        zpp.refresh_secondary(secs[j], layer[j * s:(j + 1) * s], stream=copy,
                              wait_before=primary_ready)
        zpp.quantize_blockwise_i8(secs[j], codes[j], scales[j], block=B, stream=copy,
                                  done_after=quant_done[j])
    out = empty_dev(N, np.uint16, fill=0x5A5A)
    zpp.dequant_gather_layer(codes, scales, s, N, out, block=B, stream=comm,
                             wait_events=quant_done, done_after=gather_done)
    gather_done.synchronize()
    torch.cuda.synchronize()

    ranks, ref_layer, ref_secs, ref_quants, ref_out = oracle_tiny_pipeline(hp, wl)
    for r in range(P):
        p, m, v = states[r]
        got = (to_host(p, np.float32), to_host(m, np.float32), to_host(v, np.float32),
               to_host(layer[r * n:(r + 1) * n], np.uint16))
        assert_adam_close(got, ranks[r], hp["lr"], "rank %d" % r)
    glayer = to_host(layer, np.uint16)
    same_blocks = []
    for j in range(P2):
        gsec = to_host(secs[j], np.uint16)
        assert_bits_equal(gsec, glayer[j * s:(j + 1) * s], "secondary %d = its slice" % j)
        same_blocks.append(assert_downstream(gsec, ref_secs[j], to_host(codes[j], np.int8),
                                             to_host(scales[j], np.float32), ref_quants[j][0],
                                             ref_quants[j][1], B, "shard %d" % j))
    same = np.concatenate(same_blocks)
    gout = to_host(out, np.uint16).reshape(-1, B)
    assert_bits_equal(gout[same], ref_out.reshape(-1, B)[same], "gathered layer")


def independent_streams(zpp, tries=8):
    """Two streams that the device runs side by side.  A process has a few
    hardware queues (4 by default) and two HIP streams can share one, in
    which case the device runs their work in submission order and no race
    can show.  A pair counts as independent when an event recorded on the
    second stream completes while the first is held by a bounded spin."""
    import time
    for _ in range(tries):
        a, b = torch.cuda.Stream(), torch.cuda.Stream()
        with torch.cuda.stream(a):
            torch.cuda._sleep(50_000_000)
        ev = zpp.Event().record(b)
        t0 = time.perf_counter()
        while not ev.query() and time.perf_counter() - t0 < 0.005:
            pass
        free = ev.query()
        busy = not zpp.Event().record(a).query()  # the spin still runs
        torch.cuda.synchronize()
        if free and busy:
            return a, b
    pytest.skip("no two streams of this process run side by side")


class RaceSetup:
    """Shard 0 is refreshed from `src` and quantized on the copy stream behind
    a long device-side spin; the gather of shard 0 and a peer shard runs on the
    comm stream.  The secondary starts as NaN poison, standing in for the
    uninitialised torch.empty buffer of the paper's allocation."""

    def __init__(self, zpp, s=1 << 20, B=256):
        self.zpp, self.s, self.B = zpp, s, B
        src = synth.bf16_weights(s, 90, 0)
        peer = synth.bf16_weights(s, 90, 1)
        pc, ps = oracle.quantize_blockwise_i8(peer, B)
        sc, ss = oracle.quantize_blockwise_i8(src, B)
        self.expect = oracle.dequant_gather_layer([sc, pc], [ss, ps], s, B, 2 * s)
        self.tsrc, self.tpc, self.tps = to_dev(src), to_dev(pc), to_dev(ps)
        self.copy, self.comm = independent_streams(zpp)
        self.sec = empty_dev(s, np.uint16)
        self.codes = empty_dev(s, np.int8)
        self.scales = empty_dev(s // B, np.float32)
        self.out = empty_dev(2 * s, np.uint16)
        self.done = zpp.Event()

    def run(self, fixed, spin_cycles=100_000_000):
        """One race: poison every buffer, then the spin, refresh and
        quantization on the copy stream and the gather on the comm stream,
        which waits on the quantization's event only when `fixed`."""
        zpp, B, s = self.zpp, self.B, self.s
        self.sec.fill_(0x7FC0)
        self.codes.fill_(0)
        self.scales.fill_(float("nan"))
        self.out.fill_(0)
        torch.cuda.synchronize()
        with torch.cuda.stream(self.copy):
            torch.cuda._sleep(spin_cycles)  # bounded spin kernel: the copy is still queued
        zpp.refresh_secondary(self.sec, self.tsrc, stream=self.copy)
        zpp.quantize_blockwise_i8(self.sec, self.codes, self.scales, block=B, stream=self.copy,
                                  done_after=self.done)
        zpp.dequant_gather_layer([self.codes, self.tpc], [self.scales, self.tps], s, 2 * s,
                                 self.out, block=B, stream=self.comm,
                                 wait_events=[self.done] if fixed else [])
        torch.cuda.synchronize()
        return to_host(self.out, np.uint16)


def test_fix_orders_gather_after_refresh(zpp):
    """With the event wait (the paper's fix) the gather is exact, every time,
    over 100 races in which the copy is held back behind a spin."""
    race = RaceSetup(zpp)
    for rep in range(100):
        assert_bits_equal(race.run(fixed=True), race.expect, "gather after the fix, race %d" % rep)


def test_serialized_launches_give_the_same_result(zpp):
    """With every kernel launch serialized by the runtime
    (AMD_SERIALIZE_KERNEL=3: each launch waits for the previous work and is
    waited for) the fixed path must still agree with the oracle: the smoke
    pass (Adam, refresh and quantization on two streams, the gather on a
    third after the event) runs in one child process with that setting."""
    import os
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    env = dict(os.environ, AMD_SERIALIZE_KERNEL="3")
    res = subprocess.run([sys.executable, "-c", "import __graft_entry__ as g; g.smoke()"],
                         cwd=root, env=env, capture_output=True, text=True, timeout=300)
    assert res.returncode == 0, res.stdout[-2000:] + res.stderr[-2000:]
    assert "smoke ok" in res.stdout


def test_race_without_the_fix_reads_poison(zpp):
    """Without the wait the gather runs while the copy is still queued behind
    the spin and reads the poisoned shard: NaN in the gathered layer, as the
    paper reports for stock hpZ."""
    race = RaceSetup(zpp)
    got = race.run(fixed=False)
    s = race.s
    nan = (got & 0x7FFF) > 0x7F80
    assert nan[:s].mean() > 0.99, "the racy gather did not see the poison"
    assert_bits_equal(got[s:], race.expect[s:], "peer shard")


def test_iterations_with_buffer_reuse(zpp):
    """Three iterations reusing the same secondary, codes and scale buffers:
    each refresh waits for the new primary and for the previous gather
    (write-after-read), each gather for the quantize; every iteration's state
    and gathered layer is checked against the oracle's own trajectory."""
    hp = f32hp(TINY.adam)
    n = 1 << 18
    B = 256
    P2 = 2
    s = n  # the local shard is this rank's primary; the peer shard is settled
    compute, copy, comm = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    p0 = synth.master_weights(n, 91)
    tp, tm, tv = to_dev(p0), torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    prim = empty_dev(n, np.uint16)
    sec = empty_dev(s, np.uint16, fill=0x7FC0)
    codes = empty_dev(s, np.int8)
    scales = empty_dev(s // B, np.float32)
    peer = synth.bf16_weights(s, 91, 1)
    pc, ps = oracle.quantize_blockwise_i8(peer, B)
    tpc, tps = to_dev(pc), to_dev(ps)
    out = empty_dev(P2 * s, np.uint16)
    ev_prim, ev_refresh, ev_quant, ev_gather = zpp.Event(), zpp.Event(), zpp.Event(), zpp.Event()
    grads = [synth.gradients(n, 91, it=t) for t in range(1, 4)]
    dgrads = [to_dev(g) for g in grads]
    torch.cuda.synchronize()
    snaps = []
    for t in range(1, 4):
        if t > 1:
            zpp.stream_wait(compute, ev_refresh)  # the last refresh has read the primary
        zpp.adam_partition_step(tp, tm, tv, dgrads[t - 1], prim, step=t, stream=compute, **hp)
        ev_prim.record(compute)
        if t > 1:
            zpp.stream_wait(copy, ev_gather)  # the last gather has read codes and scales
        zpp.refresh_secondary(sec, prim, stream=copy, wait_before=ev_prim, done_after=ev_refresh)
        zpp.quantize_blockwise_i8(sec, codes, scales, block=B, stream=copy, done_after=ev_quant)
        zpp.dequant_gather_layer([codes, tpc], [scales, tps], s, P2 * s, out, block=B,
                                 stream=comm, wait_events=[ev_quant], done_after=ev_gather)
        snap = empty_dev(P2 * s, np.uint16)
        with torch.cuda.stream(comm):
            snap.copy_(out)
        snaps.append(snap)
    torch.cuda.synchronize()

    rp, rm, rv = p0, np.zeros(n, np.float32), np.zeros(n, np.float32)
    mt = MomentTolerance()
    for t in range(1, 4):
        tau_m = mt.step((rp, rm, rv), grads[t - 1], hp)
        rp, rm, rv, rb = oracle.adam_step(rp, rm, rv, grads[t - 1], step=t, **hp)
        rc, rs = oracle.quantize_blockwise_i8(rb, B)
        r_out = oracle.dequant_gather_layer([rc, pc], [rs, ps], s, B, P2 * s)
        g_out = to_host(snaps[t - 1], np.uint16)
        # the peer half is exact every iteration
        assert_bits_equal(g_out[s:], r_out[s:], "peer half, iteration %d" % t)
        # the local half is the dequantized primary of this iteration
        d = np.abs(g_out[:s].view(np.int16).astype(np.int32) - r_out[:s].view(np.int16))
        assert (d == 0).mean() > 0.99, "iteration %d" % t
    got = (to_host(tp, np.float32), to_host(tm, np.float32), to_host(tv, np.float32),
           to_host(prim, np.uint16))
    assert_adam_close(got, (rp, rm, rv, rb), hp["lr"], "after 3 iterations",
                      m_tau=tau_m)
    same = assert_downstream(to_host(prim, np.uint16), rb, to_host(codes, np.int8),
                             to_host(scales, np.float32), rc, rs, B, "last iteration")
    last = to_host(snaps[-1], np.uint16)[:s].reshape(-1, B)
    assert_bits_equal(last[same], r_out[:s].reshape(-1, B)[same], "last gathered layer")


def test_pipeline_modes_agree(zpp):
    """Separate kernels or the fused one, the refresh and quantization as two
    kernels or one pass, on three streams ordered by a device event or by a
    host wait, or on one stream in path order, or switching between three
    streams and one from one iteration to the next: from the same inputs,
    three iterations end in bit-identical state, codes and gathered layer."""
    from paper_2407_01614_amd.pipeline import PartitionPipeline
    from paper_2407_01614_amd.workloads import Workload
    wl = Workload(name="small", cfg_id=9, n=1 << 20, layer_elems=8 * (1 << 17) - 1000,
                  secondary_world=8, world=8)
    p0 = synth.master_weights(wl.n, wl.cfg_id)
    g0 = synth.gradients(wl.n, wl.cfg_id)
    peers = [oracle.quantize_blockwise_i8(synth.bf16_weights(wl.shard_elems, wl.cfg_id, j + 1),
                                          wl.block) for j in range(wl.secondary_world - 1)]
    results = {}
    modes = [(fused, sync, (3, 3, 3), False) for fused in (False, True)
             for sync in ("event", "host")]
    modes += [(False, "event", (1, 1, 1), False), (True, "event", (1, 1, 1), False),
              (False, "event", (3, 1, 3), False), (True, "event", (1, 3, 1), False)]
    # the refresh and the quantization as one pass
    modes += [(False, "event", (3, 3, 3), True), (False, "host", (3, 3, 3), True),
              (False, "event", (1, 1, 1), True), (False, "event", (1, 3, 1), True)]
    for fused, sync, per_step, fuse_copy in modes:
        pipe = PartitionPipeline(wl, fused=fused, sync=sync, streams=per_step[0],
                                 fuse_copy=fuse_copy)
        pipe.load(p0, g0, [q[0] for q in peers], [q[1] for q in peers])
        for k in per_step:
            pipe.streams = k
            pipe.step()
        pipe.wait()
        results[(fused, sync, per_step, fuse_copy)] = [
            t.cpu().numpy().copy() for t in (pipe.master, pipe.exp_avg, pipe.exp_avg_sq,
                                             pipe.primary, pipe.secondary, pipe.codes,
                                             pipe.scales, pipe.out)]
    ref = results[(False, "event", (3, 3, 3), False)]
    for key, res in results.items():
        for i, (a, b) in enumerate(zip(res, ref)):
            assert_bits_equal(a.view(np.uint8), b.view(np.uint8), "%s output %d" % (key, i))
    # every output of the reference mode against the oracle: the Adam state
    # after three steps (the same gradient each step), the secondary, the
    # codes and scales (the oracle's quantization of the GPU's primary:
    # identical inputs) and the whole gathered layer
    hp = f32hp(wl.adam)
    s, B = wl.shard_elems, wl.block
    rp, rm, rv = p0, np.zeros(wl.n, np.float32), np.zeros(wl.n, np.float32)
    mt = MomentTolerance()
    for t in range(1, 4):
        tau_m = mt.step((rp, rm, rv), g0, hp)
        rp, rm, rv, rb = oracle.adam_step(rp, rm, rv, g0, step=t, **hp)
    gp, gm, gv, gb, gsec, gc, gs, gout = ref
    assert_adam_close((gp, gm, gv, gb.view(np.uint16)), (rp, rm, rv, rb), hp["lr"],
                      "reference mode after 3 steps", m_tau=tau_m)
    assert_bits_equal(gsec.view(np.uint16), gb.view(np.uint16), "secondary = primary")
    rc, rs = oracle.quantize_blockwise_i8(gb.view(np.uint16), B)
    assert_bits_equal(gc, rc, "codes")
    assert_bits_equal(gs, rs, "scales")
    expect = oracle.dequant_gather_layer([rc[:s]] + [q[0] for q in peers],
                                         [rs[:s // B]] + [q[1] for q in peers], s, B,
                                         wl.layer_elems)
    assert_bits_equal(gout.view(np.uint16), expect, "gathered layer")


@pytest.mark.parametrize("layers", [4, 5])
def test_step_gathers_every_layer(zpp, layers):
    """A step whose backward pass gathers `layers` layers, cycling over two
    stored layers (local shard k at codes [k s, (k+1) s), its own peer
    shards): every gather runs (one timed launch each), one stream and three
    streams end bit-identical, and the layer gathered last equals the oracle's
    gather of that stored layer's shards."""
    from paper_2407_01614_amd.pipeline import PartitionPipeline
    from paper_2407_01614_amd.workloads import Workload
    wl = Workload(name="small-layers", cfg_id=13, n=1 << 20, layer_elems=4 * (1 << 17) - 1000,
                  secondary_world=4, world=4, layers_gathered=layers, distinct_layers=2)
    s, B, P2 = wl.shard_elems, wl.block, wl.secondary_world
    assert wl.distinct_layers * s <= wl.n
    p0 = synth.master_weights(wl.n, wl.cfg_id)
    g0 = synth.gradients(wl.n, wl.cfg_id)
    peers = [[oracle.quantize_blockwise_i8(synth.bf16_weights(s, wl.cfg_id, j + 1, it=k), B)
              for j in range(P2 - 1)] for k in range(wl.distinct_layers)]
    outs = {}
    for streams in (1, 3):
        pipe = PartitionPipeline(wl, streams=streams)
        pipe.load(p0, g0)
        for k in range(wl.distinct_layers):
            pipe.load_layer_peers(k, [q[0] for q in peers[k]], [q[1] for q in peers[k]])
        pipe.step()
        pipe.enable_timing()
        pipe.step()
        pipe.wait()
        assert len(pipe.kernel_times_ms()["gather"]) == layers
        pipe.timing = None
        k_last = (layers - 1) % wl.distinct_layers
        codes = to_host(pipe.codes, np.int8)[k_last * s:(k_last + 1) * s]
        scales = to_host(pipe.scales, np.float32)[k_last * s // B:(k_last + 1) * s // B]
        expect = oracle.dequant_gather_layer([codes] + [q[0] for q in peers[k_last]],
                                             [scales] + [q[1] for q in peers[k_last]], s, B,
                                             wl.layer_elems)
        got = to_host(pipe.out, np.uint16)
        assert_bits_equal(got, expect, "layer %d gathered last, %d stream(s)" % (k_last, streams))
        outs[streams] = [t.cpu().numpy().copy() for t in (pipe.master, pipe.primary, pipe.codes,
                                                          pipe.out)]
        del pipe
    for a, b in zip(outs[1], outs[3]):
        assert_bits_equal(a.view(np.uint8), b.view(np.uint8), "one stream vs three")


def test_pipeline_with_qgz_receive(zpp):
    """The qgZ receive at the start of each step: the mean of 8 int4 copies of
    the partition's gradient (quantized by the oracle, as the senders would)
    becomes the gradient of the Adam step.  The reduced gradient is bit-equal
    to the oracle's, and two steps follow the oracle's Adam on it."""
    from paper_2407_01614_amd.pipeline import PartitionPipeline
    from paper_2407_01614_amd.workloads import Workload
    wl = Workload(name="small-qgz", cfg_id=12, n=(1 << 19) + 40, layer_elems=4 * (1 << 17),
                  secondary_world=4, world=4)
    P = 8
    srcs = [synth.gradients(wl.n, wl.cfg_id, q) for q in range(P)]
    quants = [oracle.quantize_blockwise_i4(x, wl.block) for x in srcs]
    pipe = PartitionPipeline(wl, qgz_sources=P)
    peers = [oracle.quantize_blockwise_i8(synth.bf16_weights(wl.shard_elems, wl.cfg_id, j + 1),
                                          wl.block) for j in range(wl.secondary_world - 1)]
    p0 = synth.master_weights(wl.n, wl.cfg_id)
    pipe.load(p0, np.zeros(wl.n, np.float32), [q[0] for q in peers], [q[1] for q in peers])
    for q, (c, sc) in enumerate(quants):
        pipe.exchange.codes[q].copy_(torch.from_numpy(c))
        pipe.exchange.scales[q].copy_(torch.from_numpy(sc))
    torch.cuda.synchronize()
    pipe.step()
    pipe.step()
    pipe.wait()
    mean = float(np.float32(1.0 / P))
    g = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], wl.n, wl.block,
                                 mean)
    assert_bits_equal(to_host(pipe.grad, np.float32), g, "reduced gradient")
    hp = f32hp(wl.adam)
    z = np.zeros(wl.n, np.float32)
    mt = MomentTolerance()
    mt.step((p0, z, z), g, hp)
    r1 = oracle.adam_step(p0, z, z, g, step=1, **hp)
    tau_m = mt.step(r1[:3], g, hp)
    r2 = oracle.adam_step(r1[0], r1[1], r1[2], g, step=2, **hp)
    got = (to_host(pipe.master, np.float32), to_host(pipe.exp_avg, np.float32),
           to_host(pipe.exp_avg_sq, np.float32), to_host(pipe.primary, np.uint16))
    assert_adam_close(got, r2, hp["lr"], "after 2 steps", m_tau=tau_m)


@pytest.mark.parametrize("streams", [1, 3])
@pytest.mark.parametrize("fuse", [False, True], ids=["reduce", "fused-receive"])
def test_pipeline_with_qgz_send(zpp, streams, fuse):
    """Each step opens with the int4 quantization of this rank's gradient
    into the exchange's send buffer (the oracle's quantization of it, bit for
    bit, after every step), then receives the 8 copies of an interleaved
    receive buffer (the oracle's quantizations of 8 ranks' gradients,
    written at set-up): two steps follow the oracle's Adam on the oracle's
    mean of the 8 copies (the separate reduce's gradient bit for bit)."""
    from paper_2407_01614_amd.pipeline import PartitionPipeline
    from paper_2407_01614_amd.workloads import Workload
    wl = Workload(name="small-qgz-send", cfg_id=15, n=(1 << 19) + 40, layer_elems=4 * (1 << 17),
                  secondary_world=4, world=4)
    P, B = 8, wl.block
    srcs = [synth.gradients(wl.n, wl.cfg_id, q) for q in range(P)]
    quants = [oracle.quantize_blockwise_i4(x, B) for x in srcs]
    own = synth.gradients(wl.n, wl.cfg_id, 99)
    pipe = PartitionPipeline(wl, qgz_sources=P, qgz_interleaved=True, streams=streams,
                             fuse_receive=fuse)
    peers = [oracle.quantize_blockwise_i8(synth.bf16_weights(wl.shard_elems, wl.cfg_id, j + 1),
                                          B) for j in range(wl.secondary_world - 1)]
    p0 = synth.master_weights(wl.n, wl.cfg_id)
    pipe.load(p0, np.zeros(wl.n, np.float32), [q[0] for q in peers], [q[1] for q in peers])
    for q in range(P):
        pipe.exchange.quantize(q, to_dev(srcs[q]))
    pipe.send_grad = to_dev(own)
    torch.cuda.synchronize()
    assert "quant_i4" in pipe.kernel_bytes()
    rc, rs = oracle.quantize_blockwise_i4(own, B)
    for t in range(2):
        pipe.step()
        pipe.wait()
        assert_bits_equal(pipe.exchange.send_codes.cpu().numpy(), rc, "sent codes, step %d" % t)
        assert_bits_equal(to_host(pipe.exchange.send_scales, np.float32), rs,
                          "sent scales, step %d" % t)
        pipe.exchange.send_codes.fill_(0x77)  # the next step must write them again
    got = deinterleave(pipe.exchange.codes.cpu().numpy(), to_host(pipe.exchange.scales,
                                                                  np.float32), wl.n, B, P)
    for q in range(P):
        assert_bits_equal(got[q][0], quants[q][0], "codes of source %d" % q)
        assert_bits_equal(got[q][1], quants[q][1], "scales of source %d" % q)
    mean = float(np.float32(1.0 / P))
    g = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], wl.n, B, mean)
    if not fuse:
        assert_bits_equal(to_host(pipe.grad, np.float32), g, "reduced gradient")
    hp = f32hp(wl.adam)
    z = np.zeros(wl.n, np.float32)
    mt = MomentTolerance()
    mt.step((p0, z, z), g, hp)
    r1 = oracle.adam_step(p0, z, z, g, step=1, **hp)
    tau_m = mt.step(r1[:3], g, hp)
    r2 = oracle.adam_step(r1[0], r1[1], r1[2], g, step=2, **hp)
    got = (to_host(pipe.master, np.float32), to_host(pipe.exp_avg, np.float32),
           to_host(pipe.exp_avg_sq, np.float32), to_host(pipe.primary, np.uint16))
    assert_adam_close(got, r2, hp["lr"], "after 2 steps", m_tau=tau_m)


def deinterleave(codes, scales, n, block, P):
    """The P sources' (codes, scales) out of an interleaved receive buffer."""
    nb = -(-n // block)
    half = block // 2
    c = codes[:nb * P * half].reshape(nb, P, half)
    s = scales[:nb * P].reshape(nb, P)
    return [(c[:, q, :].ravel()[:(n + 1) // 2].copy(), s[:, q].copy()) for q in range(P)]


@pytest.mark.parametrize("streams", [1, 3])
def test_pipeline_fused_receive_equals_separate(zpp, streams):
    """The qgZ receive fused into the partition step (no gradient buffer
    written), alone or inside the single pass of step, refresh and
    quantization, leaves the pipeline in the same state as the separate
    dequantize-and-reduce followed by the step, bit for bit, over two steps;
    the timed kernels are the ones each arrangement runs."""
    from paper_2407_01614_amd.pipeline import PartitionPipeline
    from paper_2407_01614_amd.workloads import Workload
    wl = Workload(name="small-qgz-fused", cfg_id=14, n=(1 << 19) + 40, layer_elems=4 * (1 << 17),
                  secondary_world=4, world=4)
    P = 8
    quants = [oracle.quantize_blockwise_i4(synth.gradients(wl.n, wl.cfg_id, q), wl.block)
              for q in range(P)]
    peers = [oracle.quantize_blockwise_i8(synth.bf16_weights(wl.shard_elems, wl.cfg_id, j + 1),
                                          wl.block) for j in range(wl.secondary_world - 1)]
    p0 = synth.master_weights(wl.n, wl.cfg_id)
    results = []
    expect = {(False, False): {"reduce_i4", "adam", "refresh", "quant", "gather"},
              (False, True): {"receive_adam", "refresh", "quant", "gather"},
              (True, False): {"reduce_i4", "fused", "gather"},
              (True, True): {"fused_receive", "gather"}}
    for fused, fuse in expect:
        pipe = PartitionPipeline(wl, qgz_sources=P, streams=streams, fused=fused,
                                 fuse_receive=fuse)
        pipe.load(p0, np.zeros(wl.n, np.float32), [q[0] for q in peers], [q[1] for q in peers])
        for q, (c, sc) in enumerate(quants):
            pipe.exchange.codes[q].copy_(torch.from_numpy(c))
            pipe.exchange.scales[q].copy_(torch.from_numpy(sc))
        torch.cuda.synchronize()
        pipe.step()
        pipe.enable_timing()
        pipe.step()
        pipe.wait()
        assert set(pipe.kernel_times_ms()) == expect[(fused, fuse)]
        results.append([t.cpu().numpy().copy() for t in (pipe.master, pipe.exp_avg,
                                                         pipe.exp_avg_sq, pipe.primary,
                                                         pipe.secondary, pipe.codes, pipe.scales,
                                                         pipe.out)])
        del pipe
    for other in results[1:]:
        for i, (a, b) in enumerate(zip(other, results[0])):
            assert_bits_equal(a.view(np.uint8), b.view(np.uint8), "output %d" % i)


@pytest.mark.parametrize("fused,fuse", [(False, False), (True, False), (False, True),
                                        (True, True)],
                         ids=["reduce-step", "reduce-fused", "receive-step", "single-pass"])
def test_pipeline_interleaved_receive_equals_separate(zpp, fused, fuse):
    """The pipeline with its 8 int4 copies in one interleaved receive buffer
    (each quantized into its slots on the device) ends two steps in the same
    state as with the oracle's copies in separate arrays, bit for bit, with
    the receive as its own dequantize-and-reduce kernel or fused."""
    from paper_2407_01614_amd.pipeline import PartitionPipeline
    from paper_2407_01614_amd.workloads import Workload
    wl = Workload(name="small-qgz-il", cfg_id=15, n=(1 << 19) + 40, layer_elems=4 * (1 << 17),
                  secondary_world=4, world=4)
    P = 8
    srcs = [synth.gradients(wl.n, wl.cfg_id, q) for q in range(P)]
    peers = [oracle.quantize_blockwise_i8(synth.bf16_weights(wl.shard_elems, wl.cfg_id, j + 1),
                                          wl.block) for j in range(wl.secondary_world - 1)]
    p0 = synth.master_weights(wl.n, wl.cfg_id)
    results = []
    for il in (False, True):
        pipe = PartitionPipeline(wl, qgz_sources=P, fused=fused, fuse_receive=fuse,
                                 qgz_interleaved=il)
        pipe.load(p0, np.zeros(wl.n, np.float32), [q[0] for q in peers], [q[1] for q in peers])
        for q, x in enumerate(srcs):
            if il:
                pipe.exchange.quantize(q, torch.from_numpy(x).cuda())
            else:
                c, sc = oracle.quantize_blockwise_i4(x, wl.block)
                pipe.exchange.codes[q].copy_(torch.from_numpy(c))
                pipe.exchange.scales[q].copy_(torch.from_numpy(sc))
        torch.cuda.synchronize()
        pipe.step()
        pipe.step()
        pipe.wait()
        results.append([t.cpu().numpy().copy() for t in (pipe.master, pipe.exp_avg,
                                                         pipe.exp_avg_sq, pipe.primary,
                                                         pipe.secondary, pipe.codes, pipe.scales,
                                                         pipe.out)])
        del pipe
    for i, (a, b) in enumerate(zip(results[1], results[0])):
        assert_bits_equal(a.view(np.uint8), b.view(np.uint8), "output %d" % i)

