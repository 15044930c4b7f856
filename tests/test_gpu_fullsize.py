"""Parity at full size, in the launch configuration the benchmark times.

The full Llama-2-13B rank partition (203,372,880 elements) and layer
(317,204,480 elements over 8 shards), and the padded Falcon-7B layer, run
through the same entry points with the same sizes as the benchmark, so the
kernels and grids are the ones it times.  The oracle checks a sample of
outputs it can compute one by one (elementwise Adam, whole quantization
blocks, whole gathered blocks); properties that hold at any size are checked
on everything.  Inputs are drawn on the device by the seeded generators; the
sampled inputs are copied to the host before any kernel touches them.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2407_01614_amd import synth
from paper_2407_01614_amd.pipeline import PartitionPipeline
from paper_2407_01614_amd.workloads import WORKLOADS
from parity import MomentTolerance, assert_adam_close, assert_bits_equal

pytestmark = pytest.mark.gpu

WL = WORKLOADS["llama-2-13b"]
F7 = WORKLOADS["falcon-7b-layer"]
NSAMPLE = 1 << 20
NBLOCKS = 4096


@pytest.fixture(scope="module")
def zpp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2407_01614_amd import zpp as mod
    return mod


def f32hp(hp):
    return {k: float(np.float32(v)) for k, v in hp.items()}


def sample_indices(n, k, seed):
    g = np.random.default_rng(seed)
    idx = np.unique(np.concatenate([g.integers(0, n, size=k), np.arange(4096),
                                    np.arange(n - 4096, n)]))
    return torch.from_numpy(idx).cuda()


def host(t, idx, dtype):
    return t.index_select(0, idx).cpu().numpy().view(dtype)


def test_fullsize_adam_two_steps(zpp):
    n = WL.n
    hp = f32hp(WL.adam)
    p = synth.device_normal_f32(n, synth.WEIGHT_STD, WL.cfg_id, synth.KIND_MASTER)
    g1 = synth.device_normal_f32(n, synth.GRAD_STD, WL.cfg_id, synth.KIND_GRAD, it=1)
    g2 = synth.device_normal_f32(n, synth.GRAD_STD, WL.cfg_id, synth.KIND_GRAD, it=2)
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    out = torch.empty(n, dtype=torch.int16, device="cuda")
    idx = sample_indices(n, NSAMPLE, 1)
    p0, gh1, gh2 = host(p, idx, np.float32), host(g1, idx, np.float32), host(g2, idx, np.float32)
    torch.cuda.synchronize()
    zpp.adam_partition_step(p, m, v, g1, out, step=1, **hp)
    torch.cuda.synchronize()
    got1 = tuple(host(t, idx, d) for t, d in ((p, np.float32), (m, np.float32),
                                              (v, np.float32), (out, np.uint16)))
    zpp.adam_partition_step(p, m, v, g2, out, step=2, **hp)
    torch.cuda.synchronize()
    got2 = tuple(host(t, idx, d) for t, d in ((p, np.float32), (m, np.float32),
                                              (v, np.float32), (out, np.uint16)))
    z = np.zeros_like(p0)
    r1 = oracle.adam_step(p0, z, z, gh1, step=1, **hp)
    assert_adam_close(got1, r1, hp["lr"], "step 1")
    r2 = oracle.adam_step(r1[0], r1[1], r1[2], gh2, step=2, **hp)
    mt = MomentTolerance()
    mt.step((p0, z, z), gh1, hp)
    assert_adam_close(got2, r2, hp["lr"], "step 2", steps=2, m_tau=mt.step(r1[:3], gh2, hp))
    # properties on everything: finite, bf16 is the rounding of the master
    assert torch.isfinite(p).all() and torch.isfinite(v).all() and (v >= 0).all()
    hi = (p.view(torch.int32) >> 16).to(torch.int16)
    d = (out.to(torch.int32) - hi.to(torch.int32))
    assert int(d.min()) >= 0 and int(d.max()) <= 1  # round-to-nearest of the same value


def block_sample(nblocks, k, seed):
    g = np.random.default_rng(seed)
    return np.unique(np.concatenate([g.integers(0, nblocks - 1, size=k), [0, nblocks - 2]]))


def test_fullsize_quantize(zpp):
    n, B = WL.n, WL.block
    nb = (n + B - 1) // B
    x = synth.device_bf16_weights(n, WL.cfg_id, rank=0)
    kb = block_sample(nb, NBLOCKS, 2)  # whole blocks; the short last block separately
    eidx = torch.from_numpy((kb[:, None] * B + np.arange(B)[None, :]).ravel()).cuda()
    xs = host(x, eidx, np.uint16)
    tail = x[(nb - 1) * B:].cpu().numpy().view(np.uint16)
    assert tail.size == n - (nb - 1) * B == 80
    codes = torch.empty(n, dtype=torch.int8, device="cuda")
    scales = torch.empty(nb, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    zpp.quantize_blockwise_i8(x, codes, scales, block=B)
    torch.cuda.synchronize()
    rc, rs = oracle.quantize_blockwise_i8(xs, B)
    assert_bits_equal(host(codes, eidx, np.int8), rc, "sampled blocks codes")
    assert_bits_equal(host(scales, torch.from_numpy(kb).cuda(), np.float32), rs,
                      "sampled blocks scales")
    tc, ts = oracle.quantize_blockwise_i8(tail, B)
    assert_bits_equal(codes[(nb - 1) * B:].cpu().numpy(), tc, "tail codes")
    assert_bits_equal(scales[nb - 1:].cpu().numpy(), ts, "tail scale")
    # properties on everything
    assert torch.isfinite(scales).all() and (scales > 0).all()
    assert int(codes.min()) >= -127 and int(codes.max()) <= 127
    full = codes[:(nb - 1) * B].view(nb - 1, B).to(torch.int16).abs().amax(dim=1)
    assert bool((full == 127).all()), "every block's absmax element maps to +-127"


@pytest.mark.parametrize("wl", [WL, F7], ids=["llama-2-13b-layer", "falcon-7b-layer"])
def test_fullsize_gather(zpp, wl):
    N, P2, B, s = wl.layer_elems, wl.secondary_world, wl.block, wl.shard_elems
    codes = [synth.device_random_codes(s, wl.cfg_id, rank=j) for j in range(P2)]
    scales = [synth.device_random_scales(s // B, wl.cfg_id, rank=j) for j in range(P2)]
    out = torch.full((N,), 0x5A5A, dtype=torch.int16, device="cuda")
    nbl = (N + B - 1) // B  # output blocks; with a padded last shard the last one is short
    kb = block_sample(nbl, NBLOCKS, 3)
    torch.cuda.synchronize()
    zpp.dequant_gather_layer(codes, scales, s, N, out, block=B)
    torch.cuda.synchronize()
    hc = np.empty((kb.size, B), np.int8)
    hs = np.empty(kb.size, np.float32)
    per = s // B
    for i, k in enumerate(kb):
        j, kk = divmod(int(k), per)
        hc[i] = codes[j][kk * B:(kk + 1) * B].cpu().numpy()
        hs[i] = scales[j][kk].item()
    ref = oracle.dequant_blockwise_i8(hc.ravel(), hs, B)
    eidx = torch.from_numpy((kb[:, None] * B + np.arange(B)[None, :]).ravel()).cuda()
    assert_bits_equal(host(out, eidx, np.uint16), ref, "sampled gathered blocks")
    # the end of the layer, through the last (possibly padded) shard
    j_last = (N - 1) // s
    lo = j_last * s
    tail_ref = oracle.dequant_gather_layer([codes[j_last].cpu().numpy()],
                                           [scales[j_last].cpu().numpy()], s, B, N - lo)
    assert_bits_equal(out[lo:].cpu().numpy().view(np.uint16), tail_ref, "last shard")
    assert not bool(((out & 0x7FFF) > 0x7F80).any()), "NaN in the gathered layer"


@pytest.mark.parametrize("streams", [1, 3])
def test_fullsize_pipeline_properties(zpp, streams):
    """The benchmark's own pipeline (one stream, as timed; and three streams
    with event edges), two steps: the secondary is the primary bit for bit,
    the local shard of the gathered layer round-trips the primary within half
    a quantization step, and nothing is NaN."""
    pipe = PartitionPipeline(WL, streams=streams)
    pipe.load_synthetic()
    pipe.step()
    pipe.step()
    pipe.wait()
    assert torch.equal(pipe.secondary, pipe.primary)
    s, B = WL.shard_elems, WL.block
    prim = pipe.primary[:s].view(torch.int16).to(torch.int32) << 16
    pf = prim.view(torch.float32).to(torch.float64)
    of = (pipe.out[:s].to(torch.int32) << 16).view(torch.float32).to(torch.float64)
    sc = pipe.scales[:s // B].to(torch.float64).repeat_interleave(B)
    bound = sc * (0.5 + 2.0 ** -15) + of.abs() * 2.0 ** -8
    assert bool(((pf - of).abs() <= bound).all())
    assert not bool(((pipe.out & 0x7FFF) > 0x7F80).any())
    del pipe
    torch.cuda.empty_cache()


def test_fullsize_fused_step_refresh_quantize(zpp):
    """The fused kernel on the whole Llama-2-13B partition: sampled whole
    quantization blocks (and the short last block) against the oracle's Adam
    followed by its quantizer on its own primary."""
    n, B = WL.n, WL.block
    nb = (n + B - 1) // B
    hp = f32hp(WL.adam)
    p = synth.device_normal_f32(n, synth.WEIGHT_STD, WL.cfg_id, synth.KIND_MASTER)
    g = synth.device_normal_f32(n, synth.GRAD_STD, WL.cfg_id, synth.KIND_GRAD, it=1)
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    prim = torch.empty(n, dtype=torch.int16, device="cuda")
    sec = torch.empty(n, dtype=torch.int16, device="cuda")
    codes = torch.empty(n, dtype=torch.int8, device="cuda")
    scales = torch.empty(nb, dtype=torch.float32, device="cuda")
    kb = block_sample(nb, NBLOCKS, 4)
    elems = np.concatenate([(kb[:, None] * B + np.arange(B)[None, :]).ravel(),
                            np.arange((nb - 1) * B, n)])
    eidx = torch.from_numpy(elems).cuda()
    ph, gh = host(p, eidx, np.float32), host(g, eidx, np.float32)
    torch.cuda.synchronize()
    zpp.adam_step_refresh_quantize(p, m, v, g, prim, sec, codes, scales, step=1, block=B, **hp)
    torch.cuda.synchronize()
    got = tuple(host(t, eidx, d) for t, d in ((p, np.float32), (m, np.float32), (v, np.float32),
                                              (prim, np.uint16)))
    z = np.zeros_like(ph)
    rp, rm, rv, rb = oracle.adam_step(ph, z, z, gh, step=1, **hp)
    assert_adam_close(got, (rp, rm, rv, rb), hp["lr"], "fused")
    assert torch.equal(sec, prim)
    gb = got[3]
    gc = host(codes, eidx, np.int8)
    full = kb.size * B
    rc, rs = oracle.quantize_blockwise_i8(rb[:full], B)
    same = (gb[:full].reshape(-1, B) == rb[:full].reshape(-1, B)).all(axis=1)
    assert same.mean() > 0.99
    assert_bits_equal(gc[:full].reshape(-1, B)[same], rc.reshape(-1, B)[same], "sampled codes")
    gs = host(scales, torch.from_numpy(kb).cuda(), np.float32)
    assert_bits_equal(gs[same], rs[same], "sampled scales")
    tc, ts = oracle.quantize_blockwise_i8(rb[full:], B)
    if np.array_equal(gb[full:], rb[full:]):
        assert_bits_equal(gc[full:], tc, "tail codes")
        assert_bits_equal(scales[nb - 1:].cpu().numpy(), ts, "tail scale")


@pytest.mark.parametrize("name", ["llama-2-7b", "falcon-40b"])
def test_fullsize_other_workloads(zpp, name):
    """The other rank-partition workloads, through the benchmark's pipeline
    (one stream, as timed): Llama-2-7B for 2 iterations, Falcon-40B for its
    10 iterations with fresh gradients each time and 60 layer gathers per
    iteration over 2 stored layers.  The oracle follows the sampled elements' Adam state
    through every iteration; the gathered layer is checked on sampled blocks
    against the oracle's dequantization of the codes the gather read (the
    peers' codes, drawn by the seeded generator) and, for the local shard,
    by the round-trip bound."""
    wl = WORKLOADS[name]
    iters = wl.iterations if wl.iterations > 1 else 2
    hp = f32hp(wl.adam)
    n, B, s = wl.n, wl.block, wl.shard_elems
    pipe = PartitionPipeline(wl, streams=1)
    pipe.master.copy_(synth.device_normal_f32(n, synth.WEIGHT_STD, wl.cfg_id, synth.KIND_MASTER))
    pipe.exp_avg.zero_()
    pipe.exp_avg_sq.zero_()
    for k, (pcodes, pscales) in enumerate(pipe.layer_peers):
        for j in range(wl.secondary_world - 1):
            pcodes[j].copy_(synth.device_random_codes(s, wl.cfg_id, rank=64 * k + j + 1))
            pscales[j].copy_(synth.device_random_scales(s // B, wl.cfg_id, rank=64 * k + j + 1))
    idx = sample_indices(n, 1 << 18, 5)
    p = host(pipe.master, idx, np.float32)
    m = np.zeros_like(p)
    v = np.zeros_like(p)
    mt = MomentTolerance()
    for t in range(1, iters + 1):
        g = synth.device_normal_f32(n, synth.GRAD_STD, wl.cfg_id, synth.KIND_GRAD, it=t)
        pipe.grad.copy_(g)
        gh = host(g, idx, np.float32)
        del g
        pipe.step()
        pipe.wait()
        got = tuple(host(tt, idx, d) for tt, d in ((pipe.master, np.float32),
                                                   (pipe.exp_avg, np.float32),
                                                   (pipe.exp_avg_sq, np.float32),
                                                   (pipe.primary, np.uint16)))
        tau_m = mt.step((p, m, v), gh, hp)
        p, m, v, b = oracle.adam_step(p, m, v, gh, step=t, **hp)
        assert_adam_close(got, (p, m, v, b), hp["lr"], "%s iteration %d" % (name, t), steps=t,
                          m_tau=tau_m)
    assert torch.equal(pipe.secondary, pipe.primary)
    # the layer gathered last in the step (of `layers_gathered`, cycling over
    # the stored layers) is the one left in the output
    k_last = (wl.layers_gathered - 1) % wl.distinct_layers
    peer_codes, peer_scales = pipe.layer_peers[k_last]
    # peers' part of the gathered layer: sampled whole blocks of each peer
    rng = np.random.default_rng(6)
    N = wl.layer_elems
    for j in range(1, wl.secondary_world):
        lo = j * s
        valid = min(s, N - lo)
        if valid <= 0:
            continue
        kb = np.unique(rng.integers(0, valid // B, size=64))
        codes = np.concatenate([peer_codes[j - 1][k * B:(k + 1) * B].cpu().numpy() for k in kb])
        scl = peer_scales[j - 1][torch.from_numpy(kb).cuda()].cpu().numpy()
        ref = oracle.dequant_blockwise_i8(codes, scl, B)
        eidx = torch.from_numpy((lo + kb[:, None] * B + np.arange(B)[None, :]).ravel()).cuda()
        assert_bits_equal(host(pipe.out, eidx, np.uint16), ref, "%s peer %d" % (name, j))
    # local shard: round trip of the primary within half a quantization step
    lo = k_last * s
    prim = (pipe.primary[lo:lo + s].to(torch.int32) << 16).view(torch.float32).to(torch.float64)
    of = (pipe.out[:s].to(torch.int32) << 16).view(torch.float32).to(torch.float64)
    sc = pipe.scales[lo // B:(lo + s) // B].to(torch.float64).repeat_interleave(B)
    assert bool(((prim - of).abs() <= sc * (0.5 + 2.0 ** -15) + of.abs() * 2.0 ** -8).all())
    del pipe
    torch.cuda.empty_cache()
