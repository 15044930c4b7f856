"""Sizes past 2^32 elements: 64-bit indexing and the grid-stride loops that
take over once a one-shot grid would exceed its cap.  Checked on sampled
outputs against the oracle and by properties on everything."""
import numpy as np
import pytest
import torch

import oracle
from paper_2407_01614_amd import synth
from parity import assert_adam_close, assert_bits_equal

pytestmark = pytest.mark.gpu

BIG = (1 << 32) + 4099  # crosses 2^32 with a ragged tail


@pytest.fixture(scope="module")
def zpp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    free, _ = torch.cuda.mem_get_info()
    if free < 120 * (1 << 30):
        pytest.skip("needs about 100 GiB of free device memory")
    from paper_2407_01614_amd import zpp as mod
    return mod


def sample_idx(n, seed, k=1 << 16):
    g = np.random.default_rng(seed)
    idx = np.unique(np.concatenate([g.integers(0, n, size=k), np.arange(1024),
                                    np.arange((1 << 32) - 1024, (1 << 32) + 1024),
                                    np.arange(n - 1024, n)]))
    return torch.from_numpy(idx).cuda()


def test_refresh_past_4g(zpp):
    src = synth.device_bf16_weights(BIG, 100)
    dst = torch.empty_like(src)
    zpp.refresh_secondary(dst, src)
    torch.cuda.synchronize()
    assert torch.equal(dst, src)
    del src, dst
    torch.cuda.empty_cache()


def test_adam_past_4g(zpp):
    n = BIG
    hp = {k: float(np.float32(v)) for k, v in
          dict(lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1).items()}
    p = synth.device_normal_f32(n, synth.WEIGHT_STD, 101, synth.KIND_MASTER)
    g = synth.device_normal_f32(n, synth.GRAD_STD, 101, synth.KIND_GRAD)
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    out = torch.empty(n, dtype=torch.int16, device="cuda")
    idx = sample_idx(n, 1)
    ph = p.index_select(0, idx).cpu().numpy()
    gh = g.index_select(0, idx).cpu().numpy()
    zpp.adam_partition_step(p, m, v, g, out, step=1, **hp)
    torch.cuda.synchronize()
    got = tuple(t.index_select(0, idx).cpu().numpy().view(d) for t, d in
                ((p, np.float32), (m, np.float32), (v, np.float32), (out, np.uint16)))
    z = np.zeros_like(ph)
    assert_adam_close(got, oracle.adam_step(ph, z, z, gh, step=1, **hp), hp["lr"], "past 2^32")
    assert bool(torch.isfinite(p).all())
    del p, g, m, v, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("B", [256, 320])
def test_quantize_past_4g(zpp, B):
    n = BIG
    nb = (n + B - 1) // B
    x = synth.device_bf16_weights(n, 102)
    codes = torch.empty(n, dtype=torch.int8, device="cuda")
    scales = torch.empty(nb, dtype=torch.float32, device="cuda")
    zpp.quantize_blockwise_i8(x, codes, scales, block=B)
    torch.cuda.synchronize()
    g = np.random.default_rng(3)
    kb = np.unique(np.concatenate([g.integers(0, nb - 1, size=2048),
                                   [(1 << 32) // B - 1, (1 << 32) // B, nb - 2]]))
    eidx = torch.from_numpy((kb[:, None] * B + np.arange(B)[None, :]).ravel()).cuda()
    rc, rs = oracle.quantize_blockwise_i8(x.index_select(0, eidx).cpu().numpy().view(np.uint16), B)
    assert_bits_equal(codes.index_select(0, eidx).cpu().numpy(), rc, "codes")
    assert_bits_equal(scales[torch.from_numpy(kb).cuda()].cpu().numpy(), rs, "scales")
    tail = x[(nb - 1) * B:].cpu().numpy().view(np.uint16)
    tc, ts = oracle.quantize_blockwise_i8(tail, B)
    assert_bits_equal(codes[(nb - 1) * B:].cpu().numpy(), tc, "tail codes")
    assert_bits_equal(scales[nb - 1:].cpu().numpy(), ts, "tail scale")
    assert bool((scales > 0).all())
    del x, codes, scales
    torch.cuda.empty_cache()


@pytest.mark.parametrize("B,P2,s", [(256, 2, (1 << 31) + (1 << 20)),
                                    (192, 1, ((1 << 32) + 4099 + 191) // 192 * 192)],
                         ids=["2-shards", "one-shard-block-192"])
def test_gather_past_4g(zpp, B, P2, s):
    """A layer of more than 2^32 elements from 2 shards of 2^31 + 2^20, or
    from one shard past 2^32 in blocks that are not a power of two (block
    indices past 2^32 / 192 through the quotient of the block size)."""
    N = P2 * s - 777
    codes = [synth.device_random_codes(s, 103, rank=j) for j in range(P2)]
    scales = [synth.device_random_scales(s // B, 103, rank=j) for j in range(P2)]
    out = torch.empty(N, dtype=torch.int16, device="cuda")
    zpp.dequant_gather_layer(codes, scales, s, N, out, block=B)
    torch.cuda.synchronize()
    g = np.random.default_rng(4)
    per = s // B
    kb = np.unique(np.concatenate([g.integers(0, P2 * per - 1, size=1024),
                                   [per - 1, min(per, P2 * per - 2)],
                                   [(1 << 32) // B - 1, (1 << 32) // B]]))
    kb = kb[kb < P2 * per - 8]
    hc = np.concatenate([codes[k // per][(k % per) * B:(k % per + 1) * B].cpu().numpy() for k in kb])
    hs = np.array([scales[k // per][k % per].item() for k in kb], np.float32)
    ref = oracle.dequant_blockwise_i8(hc, hs, B)
    eidx = torch.from_numpy((kb[:, None] * B + np.arange(B)[None, :]).ravel()).cuda()
    assert_bits_equal(out.index_select(0, eidx).cpu().numpy().view(np.uint16), ref, "sampled")
    # the end of the layer: the last 8 blocks of the last shard reach past N
    start = P2 * s - 8 * B
    tail_ref = oracle.dequant_gather_layer([codes[-1][-(8 * B):].cpu().numpy()],
                                           [scales[-1][-8:].cpu().numpy()], 8 * B, B, N - start)
    assert_bits_equal(out[start:].cpu().numpy().view(np.uint16), tail_ref, "tail")
    del codes, scales, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("single_pass", [False, True], ids=["step", "single-pass"])
def test_receive_adam_past_4g(zpp, single_pass):
    """The qgZ receive fused into the partition step over more than 2^32
    elements from 2 int4 sources (arbitrary packed codes and scales from the
    input generator): sampled whole blocks (around 2^32 and the
    ragged tail included) against the oracle's dequantize-and-reduce followed
    by its Adam step.  The single pass also writes the secondary (equal to the
    primary everywhere) and its int8 quantization (the oracle's quantization
    of the GPU's primary on the same blocks, bit for bit)."""
    n, B, P = BIG, 256, 2
    nb = (n + B - 1) // B
    hp = {k: float(np.float32(v)) for k, v in
          dict(lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1).items()}
    # the int4 copies as the exchange would deliver them: arbitrary packed
    # codes and scales drawn by the input generator
    codes = [synth.device_random_packed_i4((n + 1) // 2, 104, rank=q) for q in range(P)]
    scales = [synth.device_random_scales(nb, 104, rank=q, lo=1e-5, hi=2e-4) for q in range(P)]
    p = synth.device_normal_f32(n, synth.WEIGHT_STD, 104, synth.KIND_MASTER)
    m = torch.zeros(n, device="cuda")
    v = torch.zeros(n, device="cuda")
    out = torch.empty(n, dtype=torch.int16, device="cuda")
    g = np.random.default_rng(5)
    kb = np.unique(np.concatenate([g.integers(0, nb - 1, size=2048),
                                   [(1 << 32) // B - 1, (1 << 32) // B, nb - 2]]))
    eidx = torch.from_numpy((kb[:, None] * B + np.arange(B)[None, :]).ravel()).cuda()
    cidx = torch.from_numpy((kb[:, None] * (B // 2) + np.arange(B // 2)[None, :]).ravel()).cuda()
    sidx = torch.from_numpy(kb).cuda()
    ph = p.index_select(0, eidx).cpu().numpy()
    hc = [c.index_select(0, cidx).cpu().numpy() for c in codes]
    hs = [s.index_select(0, sidx).cpu().numpy() for s in scales]
    tail = n - (nb - 1) * B
    tidx = torch.arange((nb - 1) * B, n, device="cuda")
    tp = p[(nb - 1) * B:].cpu().numpy()
    tc = [c[(nb - 1) * B // 2:].cpu().numpy() for c in codes]
    ts = [s[nb - 1:].cpu().numpy() for s in scales]
    if single_pass:
        sec = torch.empty(n, dtype=torch.int16, device="cuda")
        q8 = torch.empty(n, dtype=torch.int8, device="cuda")
        s8 = torch.empty(nb, dtype=torch.float32, device="cuda")
        zpp.qgz_receive_step_refresh_quantize(p, m, v, codes, scales, out, sec, q8, s8, step=1,
                                              grad_block=B, block=B, scale_out=0.5, **hp)
    else:
        zpp.qgz_receive_adam_step(p, m, v, codes, scales, out, step=1, block=B, scale_out=0.5,
                                  **hp)
    torch.cuda.synchronize()
    half = float(np.float32(0.5))
    for what, idx, p_ref, c_ref, s_ref, k, blocks in (
            ("sampled blocks", eidx, ph, hc, hs, kb.size * B, sidx),
            ("tail", tidx, tp, tc, ts, tail, torch.tensor([nb - 1], device="cuda"))):
        gr = oracle.dequant_reduce_i4(c_ref, s_ref, k, B, half)
        z = np.zeros(k, np.float32)
        got = tuple(t.index_select(0, idx).cpu().numpy().view(d) for t, d in
                    ((p, np.float32), (m, np.float32), (v, np.float32), (out, np.uint16)))
        assert_adam_close(got, oracle.adam_step(p_ref, z, z, gr, step=1, **hp), hp["lr"],
                          "receive step past 2^32, " + what)
        if single_pass:
            rc, rs = oracle.quantize_blockwise_i8(got[3], B)
            assert_bits_equal(q8.index_select(0, idx).cpu().numpy(), rc, "codes, " + what)
            assert_bits_equal(s8.index_select(0, blocks).cpu().numpy(), rs, "scales, " + what)
    if single_pass:
        assert torch.equal(sec, out)
        del sec, q8, s8
    del p, m, v, out, codes, scales
    torch.cuda.empty_cache()
