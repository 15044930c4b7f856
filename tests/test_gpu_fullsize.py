"""Parity at full size, in the launch configuration the benchmark times.

The full Llama-2-13B rank partition (203,372,880 elements) and layer
(317,204,480 elements over 8 shards), and the padded Falcon-7B layer, run
through the same entry points with the same sizes as the benchmark, so the
kernels and grids are the ones it times.  The optimizer step, the
quantization and the gather are compared with the oracle over the whole
arrays (the oracle runs on block-aligned ranges from a pool of host
threads), every element of every array, plus properties that hold at any
size; the fused kernel is compared on sampled quantization blocks.  Inputs
are drawn on the device by the seeded generators and copied to the host
before any kernel touches them.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from paper_2407_01614_amd import synth
from paper_2407_01614_amd.pipeline import PartitionPipeline
from paper_2407_01614_amd.workloads import WORKLOADS, secondary_elems
from parity import ChunkedAdam, assert_adam_close, assert_bits_equal

pytestmark = pytest.mark.gpu

WL = WORKLOADS["llama-2-13b"]
F7 = WORKLOADS["falcon-7b-layer"]
NBLOCKS = 4096


@pytest.fixture(scope="module")
def zpp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2407_01614_amd import zpp as mod
    return mod


def f32hp(hp):
    return {k: float(np.float32(v)) for k, v in hp.items()}


def host(t, idx, dtype):
    return t.index_select(0, idx).cpu().numpy().view(dtype)


def pool():
    try:
        k = len(os.sched_getaffinity(0))
    except AttributeError:
        k = os.cpu_count() or 1
    return ThreadPoolExecutor(max(1, min(16, k)))


def oracle_quantize_whole(x, B, ex):
    """The oracle's quantization of a whole array, on block-aligned ranges."""
    n = x.size
    step = max(B, -(-n // 64) // B * B)
    parts = list(ex.map(lambda a: oracle.quantize_blockwise_i8(x[a:a + step], B),
                        range(0, n, step)))
    return np.concatenate([c for c, _ in parts]), np.concatenate([sc for _, sc in parts])


def whole(t, dtype):
    return t.cpu().numpy().view(dtype)


def test_fullsize_adam_two_steps(zpp):
    """Two steps over the whole Llama-2-13B partition (203,372,880 elements),
    every element against the oracle after each; then properties on
    everything."""
    n = WL.n
    hp = f32hp(WL.adam)
    p = synth.device_normal_f32(n, synth.WEIGHT_STD, WL.cfg_id, synth.KIND_MASTER)
    g1 = synth.device_normal_f32(n, synth.GRAD_STD, WL.cfg_id, synth.KIND_GRAD, it=1)
    g2 = synth.device_normal_f32(n, synth.GRAD_STD, WL.cfg_id, synth.KIND_GRAD, it=2)
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    out = torch.empty(n, dtype=torch.int16, device="cuda")
    p0, gh1, gh2 = whole(p, np.float32), whole(g1, np.float32), whole(g2, np.float32)
    torch.cuda.synchronize()
    with pool() as ex:
        ref = ChunkedAdam(p0, hp, ex)
        for t, (g, gh) in enumerate(((g1, gh1), (g2, gh2)), start=1):
            zpp.adam_partition_step(p, m, v, g, out, step=t, **hp)
            torch.cuda.synchronize()
            ref.step(gh)
            ref.check(tuple(whole(x, d) for x, d in ((p, np.float32), (m, np.float32),
                                                     (v, np.float32), (out, np.uint16))),
                      "step %d" % t)
    # properties on everything: finite, bf16 is the rounding of the master
    assert torch.isfinite(p).all() and torch.isfinite(v).all() and (v >= 0).all()
    hi = (p.view(torch.int32) >> 16).to(torch.int16)
    d = (out.to(torch.int32) - hi.to(torch.int32))
    assert int(d.min()) >= 0 and int(d.max()) <= 1  # round-to-nearest of the same value


def block_sample(nblocks, k, seed):
    g = np.random.default_rng(seed)
    return np.unique(np.concatenate([g.integers(0, nblocks - 1, size=k), [0, nblocks - 2]]))


def test_fullsize_quantize(zpp):
    """Every block of the Llama-2-13B partition (794,427 blocks; the last
    holds 80 elements) against the oracle, bit for bit."""
    n, B = WL.n, WL.block
    nb = (n + B - 1) // B
    assert n - (nb - 1) * B == 80
    x = synth.device_bf16_weights(n, WL.cfg_id, rank=0)
    xh = x.cpu().numpy().view(np.uint16)
    codes = torch.empty(n, dtype=torch.int8, device="cuda")
    scales = torch.empty(nb, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    zpp.quantize_blockwise_i8(x, codes, scales, block=B)
    torch.cuda.synchronize()
    with pool() as ex:
        rc, rs = oracle_quantize_whole(xh, B, ex)
    assert_bits_equal(codes.cpu().numpy(), rc, "whole codes")
    assert_bits_equal(scales.cpu().numpy(), rs, "whole scales")
    # properties on everything
    assert torch.isfinite(scales).all() and (scales > 0).all()
    assert int(codes.min()) >= -127 and int(codes.max()) <= 127
    full = codes[:(nb - 1) * B].view(nb - 1, B).to(torch.int16).abs().amax(dim=1)
    assert bool((full == 127).all()), "every block's absmax element maps to +-127"


@pytest.mark.parametrize("B", [192, 2112])
def test_fullsize_quantize_blocks_not_powers_of_two(zpp, B):
    """The lane-group quantizers over the whole Llama-2-13B partition at
    blocks that are not powers of two: int8 codes and scales, alone and in
    the pass with the secondary copy, and int4 codes and scales of an fp32
    gradient of the same length, every block against the oracle, bit for
    bit."""
    n = WL.n
    nb = (n + B - 1) // B
    x = synth.device_bf16_weights(n, WL.cfg_id, rank=1)
    xh = x.cpu().numpy().view(np.uint16)
    codes = torch.empty(n, dtype=torch.int8, device="cuda")
    scales = torch.empty(nb, dtype=torch.float32, device="cuda")
    sec = torch.empty(n, dtype=torch.bfloat16, device="cuda")
    with pool() as ex:
        rc, rs = oracle_quantize_whole(xh, B, ex)
    zpp.quantize_blockwise_i8(x, codes, scales, block=B)
    torch.cuda.synchronize()
    assert_bits_equal(codes.cpu().numpy(), rc, "int8 codes B=%d" % B)
    assert_bits_equal(scales.cpu().numpy(), rs, "int8 scales B=%d" % B)
    codes.fill_(99)
    scales.fill_(-1.0)
    zpp.refresh_quantize_i8(sec, x, codes, scales, block=B)
    torch.cuda.synchronize()
    assert_bits_equal(sec.view(torch.int16).cpu().numpy().view(np.uint16), xh,
                      "secondary B=%d" % B)
    assert_bits_equal(codes.cpu().numpy(), rc, "int8 codes with the copy B=%d" % B)
    assert_bits_equal(scales.cpu().numpy(), rs, "int8 scales with the copy B=%d" % B)
    del sec, codes, x
    g = synth.device_normal_f32(n, synth.GRAD_STD, WL.cfg_id, synth.KIND_GRAD, it=3)
    c4 = torch.empty((n + 1) // 2, dtype=torch.uint8, device="cuda")
    zpp.quantize_blockwise_i4(g, c4, scales, block=B)
    torch.cuda.synchronize()
    gh = g.cpu().numpy()
    step = max(B, -(-n // 64) // B * B)
    with pool() as ex:
        parts = list(ex.map(lambda a: oracle.quantize_blockwise_i4(gh[a:a + step], B),
                            range(0, n, step)))
    assert_bits_equal(c4.cpu().numpy(), np.concatenate([c for c, _ in parts]),
                      "int4 codes B=%d" % B)
    assert_bits_equal(scales.cpu().numpy(), np.concatenate([sc for _, sc in parts]),
                      "int4 scales B=%d" % B)


@pytest.mark.parametrize("wl", [WL, F7], ids=["llama-2-13b-layer", "falcon-7b-layer"])
def test_fullsize_gather(zpp, wl):
    """The whole gathered layer (317,204,480 or 207,070,080 elements, the
    latter through a padded last shard) against the oracle, bit for bit."""
    N, P2, B, s = wl.layer_elems, wl.secondary_world, wl.block, wl.shard_elems
    codes = [synth.device_random_codes(s, wl.cfg_id, rank=j) for j in range(P2)]
    scales = [synth.device_random_scales(s // B, wl.cfg_id, rank=j) for j in range(P2)]
    out = torch.full((N,), 0x5A5A, dtype=torch.int16, device="cuda")
    torch.cuda.synchronize()
    zpp.dequant_gather_layer(codes, scales, s, N, out, block=B)
    torch.cuda.synchronize()
    hc = [c.cpu().numpy() for c in codes]
    hs = [x.cpu().numpy() for x in scales]
    with pool() as ex:
        ref = list(ex.map(lambda j: oracle.dequant_gather_layer(
            [hc[j]], [hs[j]], s, B, min(s, N - j * s)), range(P2)))
    assert_bits_equal(out.cpu().numpy().view(np.uint16), np.concatenate(ref), "whole layer")
    assert not bool(((out & 0x7FFF) > 0x7F80).any()), "NaN in the gathered layer"


@pytest.mark.parametrize("name", ["llama-2-13b", "falcon-40b"])
def test_fullsize_forward_gather(zpp, name):
    """The forward AllGather(L, P) with qwZ as one GPU carries it, end to end
    in the calls the benchmark times: a layer of bf16 weights split into the
    P ranks' primary slices (64 with a padded last one for Llama-2-13B; 128
    for Falcon-40B, gathered in two calls of 64 each writing its half), each
    slice int8-quantized by the library, then the layer gathered from all
    slices.  Against the oracle's quantization of the same slices and its
    gather of them, bit for bit: every code, every scale, the whole layer."""
    wl = WORKLOADS[name]
    N, P, B = wl.layer_elems, wl.world, wl.block
    s = oracle.secondary_shard_elems(N, P, B)
    assert s == secondary_elems(N, P, B)
    w = synth.device_bf16_weights(P * s, wl.cfg_id, rank=1000)
    w[N:] = 0  # the padding of the last slice
    codes = [torch.empty(s, dtype=torch.int8, device="cuda") for _ in range(P)]
    scales = [torch.empty(s // B, dtype=torch.float32, device="cuda") for _ in range(P)]
    out = torch.full((N,), 0x5A5A, dtype=torch.int16, device="cuda")
    wh = w.cpu().numpy().view(np.uint16)
    torch.cuda.synchronize()
    for j in range(P):
        zpp.quantize_blockwise_i8(w[j * s:(j + 1) * s], codes[j], scales[j], block=B)
    G = zpp.MAX_SHARDS
    for g0 in range(0, P, G):
        part = min(N - g0 * s, min(G, P - g0) * s)
        if part <= 0:
            continue  # a group of slices that holds only padding
        zpp.dequant_gather_layer(codes[g0:g0 + G], scales[g0:g0 + G], s, part, out[g0 * s:],
                                 block=B)
    torch.cuda.synchronize()
    hc = [c.cpu().numpy() for c in codes]
    hs = [x.cpu().numpy() for x in scales]
    del w, codes, scales
    with pool() as ex:
        ref = list(ex.map(lambda j: oracle.quantize_blockwise_i8(wh[j * s:(j + 1) * s], B),
                          range(P)))
        for j in range(P):
            assert_bits_equal(hc[j], ref[j][0], "codes of slice %d" % j)
            assert_bits_equal(hs[j], ref[j][1], "scales of slice %d" % j)
        layer = list(ex.map(lambda j: oracle.dequant_gather_layer(
            [ref[j][0]], [ref[j][1]], s, B, max(0, min(s, N - j * s))), range(P)))
    assert_bits_equal(out.cpu().numpy().view(np.uint16), np.concatenate(layer), "whole layer")
    del out
    torch.cuda.empty_cache()


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


@pytest.mark.parametrize("B", [256, 320, 4096])
def test_fullsize_fused_step_refresh_quantize(zpp, B):
    """The fused step on the whole Llama-2-13B partition (one pass at 256;
    the step with its copies, then the quantizer, at 320 and 4096): sampled
    whole quantization blocks (and the short last block) against the
    oracle's Adam followed by its quantizer on its own primary."""
    n = WL.n
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
    # a primary element may differ by one bf16 ulp where the fp32 update
    # lands near a rounding tie (within the Adam tolerance above); a block
    # of 4096 holds such an element 16 times as often as one of 256
    assert same.mean() > (0.99 if B <= 320 else 0.9)
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
    iteration over 2 stored layers.  The oracle follows the whole partition's
    Adam state through every iteration; after the last, the quantized
    secondary and the layer gathered last are compared whole, bit for bit,
    with the oracle's quantization of the GPU's primary and its gather of the
    shards that layer read."""
    wl = WORKLOADS[name]
    iters = wl.iterations if wl.iterations > 1 else 2
    hp = f32hp(wl.adam)
    n, B, s, N, P2 = wl.n, wl.block, wl.shard_elems, wl.layer_elems, wl.secondary_world
    pipe = PartitionPipeline(wl, streams=1)
    pipe.master.copy_(synth.device_normal_f32(n, synth.WEIGHT_STD, wl.cfg_id, synth.KIND_MASTER))
    pipe.exp_avg.zero_()
    pipe.exp_avg_sq.zero_()
    for k, (pcodes, pscales) in enumerate(pipe.layer_peers):
        for j in range(P2 - 1):
            pcodes[j].copy_(synth.device_random_codes(s, wl.cfg_id, rank=64 * k + j + 1))
            pscales[j].copy_(synth.device_random_scales(s // B, wl.cfg_id, rank=64 * k + j + 1))
    with pool() as ex:
        ref = ChunkedAdam(whole(pipe.master, np.float32), hp, ex)
        for t in range(1, iters + 1):
            g = synth.device_normal_f32(n, synth.GRAD_STD, wl.cfg_id, synth.KIND_GRAD, it=t)
            pipe.grad.copy_(g)
            gh = whole(g, np.float32)
            del g
            pipe.step()
            pipe.wait()
            ref.step(gh)
            del gh
        ref.check(tuple(whole(tt, d) for tt, d in ((pipe.master, np.float32),
                                                   (pipe.exp_avg, np.float32),
                                                   (pipe.exp_avg_sq, np.float32),
                                                   (pipe.primary, np.uint16))),
                  "%s after %d iterations" % (name, iters))
        del ref
        assert torch.equal(pipe.secondary, pipe.primary)
        prim = whole(pipe.primary, np.uint16)
        codes, scales = whole(pipe.codes, np.int8), whole(pipe.scales, np.float32)
        rc, rs = oracle_quantize_whole(prim, B, ex)
        assert_bits_equal(codes, rc, "%s codes" % name)
        assert_bits_equal(scales, rs, "%s scales" % name)
        # the layer gathered last in the step (of `layers_gathered`, cycling
        # over the stored layers) is the one left in the output; its local
        # shard is codes [k s, (k+1) s) of this rank's quantized secondary
        k_last = (wl.layers_gathered - 1) % wl.distinct_layers
        peer_codes, peer_scales = pipe.layer_peers[k_last]
        shard_c = [codes[k_last * s:(k_last + 1) * s]] + [whole(c, np.int8) for c in peer_codes]
        shard_s = ([scales[k_last * s // B:(k_last + 1) * s // B]]
                   + [whole(x, np.float32) for x in peer_scales])
        ref = list(ex.map(lambda j: oracle.dequant_gather_layer(
            [shard_c[j]], [shard_s[j]], s, B, min(s, N - j * s)), range(P2)))
    assert_bits_equal(whole(pipe.out, np.uint16), np.concatenate(ref), "%s layer" % name)
    del pipe
    torch.cuda.empty_cache()
