"""GPU parity of the qgZ gradient side (int4 quantization, the
dequantize-and-reduce, and the receive fused into the partition step)
against the CPU oracle and the unfused sequence, through the C ABI."""
import numpy as np
import pytest
import torch

import oracle
from paper_2407_01614_amd import synth
from paper_2407_01614_amd.workloads import WORKLOADS
from parity import (assert_adam_close, assert_bits_equal, empty_dev, first_moment_scale,
                    to_dev, to_host)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def zpp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2407_01614_amd import zpp as mod
    return mod


def u8_dev(a, pad=0):
    a = np.ascontiguousarray(a, np.uint8)
    t = torch.from_numpy(a)
    if pad:
        buf = torch.zeros(a.size + pad, dtype=torch.uint8, device="cuda")
        buf[pad:].copy_(t.cuda())
        return buf[pad:]
    return t.cuda()


def run_quant_i4(zpp, x, block, pad_src=0, pad_codes=0):
    tx = to_dev(x, pad=pad_src)
    nbytes = (x.size + 1) // 2
    cbuf = torch.full((nbytes + pad_codes,), 0xAA, dtype=torch.uint8, device="cuda")
    codes = cbuf[pad_codes:]
    scales = empty_dev((x.size + block - 1) // block, np.float32, fill=-1.0)
    zpp.quantize_blockwise_i4(tx, codes, scales, block=block)
    torch.cuda.synchronize()
    return codes.cpu().numpy(), to_host(scales, np.float32)


def grads(n, cfg, rank=0, scale=1.0):
    return synth.gradients(n, cfg, rank) * np.float32(scale)


@pytest.mark.parametrize("block", [64, 128, 192, 256, 320, 512, 960, 2048, 2112, 4032,
                                   4096])
@pytest.mark.parametrize("n", [1, 2, 7, 8, 9, 255, 256, 257, 256 * 9 + 81, 100001, 1 << 18])
def test_quant_i4_vs_oracle(zpp, block, n):
    x = grads(n, 80, n + block)
    got = run_quant_i4(zpp, x, block)
    ref = oracle.quantize_blockwise_i4(x, block)
    assert_bits_equal(got[0], ref[0], "codes n=%d block=%d" % (n, block))
    assert_bits_equal(got[1], ref[1], "scales n=%d block=%d" % (n, block))


@pytest.mark.parametrize("pads", [(1, 0), (0, 1), (4, 2)], ids=["src", "codes", "both"])
def test_quant_i4_misaligned(zpp, pads):
    x = grads(256 * 13 + 33, 81)
    got = run_quant_i4(zpp, x, 256, *pads)
    ref = oracle.quantize_blockwise_i4(x, 256)
    assert_bits_equal(got[0], ref[0], "codes")
    assert_bits_equal(got[1], ref[1], "scales")


def i4_special(block):
    rng = np.random.default_rng(82)
    parts = [np.zeros(block, np.float32)]
    b = (rng.standard_normal(block) * 1e-3).astype(np.float32); b[1] = np.inf; parts.append(b)
    b = (rng.standard_normal(block) * 1e-3).astype(np.float32); b[-1] = -np.inf; parts.append(b)
    b = (rng.standard_normal(block) * 1e-3).astype(np.float32); b[7] = np.nan; parts.append(b)
    for e in (-149, -140, -126, -110, -101, -100, -60, 0, 60, 120):
        q = rng.integers(-7, 8, size=block).astype(np.float64)
        q[rng.integers(0, block)] = -7
        parts.append((q * 2.0 ** e).astype(np.float32))
    ties = np.zeros(block, np.float32)
    ties[:9] = [7.0, 0.5, 1.5, 2.5, 3.5, -0.5, -1.5, 6.5, -6.5]
    parts.append(ties)
    parts.append((rng.standard_normal(block) * 1e-42).astype(np.float32))  # subnormal block
    parts.append(np.full(block, -0.0, np.float32))
    return np.concatenate(parts)


@pytest.mark.parametrize("block", [64, 192, 256, 1024])
@pytest.mark.parametrize("pad", [0, 1], ids=["vector", "scalar"])
def test_quant_i4_special_blocks(zpp, block, pad):
    x = i4_special(block)
    got = run_quant_i4(zpp, x, block, pad_src=pad)
    ref = oracle.quantize_blockwise_i4(x, block)
    assert_bits_equal(got[0], ref[0], "codes")
    assert_bits_equal(got[1], ref[1], "scales")


def oracle_sources(P, n, block, cfg):
    srcs = [grads(n, cfg, q, scale=1.0 + q) for q in range(P)]
    return [oracle.quantize_blockwise_i4(s, block) for s in srcs]


def run_reduce_i4(zpp, quants, n, block, scale_out, pad_out=0, pad_codes=0):
    codes = [u8_dev(c, pad=pad_codes) for c, _ in quants]
    scales = [to_dev(s) for _, s in quants]
    out = empty_dev(n, np.float32, pad=pad_out, fill=-7.0)
    zpp.dequant_reduce_i4(codes, scales, n, out, block=block, scale_out=scale_out)
    torch.cuda.synchronize()
    return to_host(out, np.float32)


@pytest.mark.parametrize("P", [1, 2, 3, 8, 13, 64])
@pytest.mark.parametrize("n", [1, 7, 8, 9, 256 * 5 + 3, 65536 + 8])
def test_dequant_reduce_i4_vs_oracle(zpp, P, n):
    block = 256
    quants = oracle_sources(P, n, block, 83 + n)
    for scale_out in (1.0, float(np.float32(1.0 / P))):
        got = run_reduce_i4(zpp, quants, n, block, scale_out)
        ref = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], n, block,
                                       scale_out)
        assert_bits_equal(got, ref, "P=%d n=%d scale_out=%g" % (P, n, scale_out))


@pytest.mark.parametrize("P,n,block", [(8, 192 * 37 + 5, 192), (3, 320 * 11 + 7, 320),
                                       (5, 4032 * 3 + 33, 4032)])
@pytest.mark.parametrize("pad_out", [0, 1], ids=["vector", "scalar"])
def test_dequant_reduce_i4_blocks_not_powers_of_two(zpp, P, n, block, pad_out):
    quants = oracle_sources(P, n, block, 85 + n)
    got = run_reduce_i4(zpp, quants, n, block, float(np.float32(1.0 / P)), pad_out=pad_out)
    ref = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], n, block,
                                   float(np.float32(1.0 / P)))
    assert_bits_equal(got, ref, "P=%d n=%d block=%d" % (P, n, block))


@pytest.mark.parametrize("pads", [(1, 0), (0, 1)], ids=["out", "codes"])
def test_dequant_reduce_i4_misaligned(zpp, pads):
    n, block, P = 256 * 11 + 5, 128, 5
    quants = oracle_sources(P, n, block, 84)
    got = run_reduce_i4(zpp, quants, n, block, 0.2, *pads)
    ref = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], n, block,
                                   float(np.float32(0.2)))
    assert_bits_equal(got, ref, "misaligned")


def test_dequant_reduce_i4_special_scales(zpp):
    n, block, P = 256 * 8, 256, 4
    quants = oracle_sources(P, n, block, 85)
    quants[1][1][2] = np.nan
    quants[2][1][3] = np.inf
    quants[3][1][4] = 0.0
    quants[0][1][5] = 1e-40
    got = run_reduce_i4(zpp, quants, n, block, 1.0)
    ref = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], n, block, 1.0)
    assert_bits_equal(got, ref, "special scales")


def test_qgz_exchange_one_partition(zpp):
    """The qgZ exchange seen by one rank: P sending ranks quantize their
    gradient of this rank's partition on the GPU, the rank reduces the P
    copies into the mean gradient; both steps bit-equal to the oracle run on
    the same fp32 gradients."""
    P, n, block = 8, 300000 + 17, 256
    srcs = [grads(n, 86, q) for q in range(P)]
    gq = [run_quant_i4(zpp, s, block) for s in srcs]
    rq = [oracle.quantize_blockwise_i4(s, block) for s in srcs]
    for q in range(P):
        assert_bits_equal(gq[q][0], rq[q][0], "source %d codes" % q)
        assert_bits_equal(gq[q][1], rq[q][1], "source %d scales" % q)
    mean = float(np.float32(1.0 / P))
    got = run_reduce_i4(zpp, gq, n, block, mean)
    ref = oracle.dequant_reduce_i4([c for c, _ in rq], [s for _, s in rq], n, block, mean)
    assert_bits_equal(got, ref, "mean gradient")
    # the quantized mean stays within the quantization error of the true mean
    true = np.mean(np.stack(srcs).astype(np.float64), axis=0)
    err_bound = np.mean(np.stack([np.repeat(s, block)[:n] for _, s in rq]), axis=0) * 0.5001
    assert np.all(np.abs(got - true) <= err_bound + 1e-12)


def test_fullsize_qgz_partition(zpp):
    """The Llama-2-13B partition (203,372,880 values) from 8 sources, in the
    configuration the benchmark times: sampled blocks against the oracle."""
    wl = WORKLOADS["llama-2-13b"]
    n, block, P = wl.n, wl.block, 8
    nb = (n + block - 1) // block
    src = [synth.device_normal_f32(n, synth.GRAD_STD, wl.cfg_id, synth.KIND_GRAD, rank=q)
           for q in range(P)]
    g = np.random.default_rng(87)
    kb = np.unique(np.concatenate([g.integers(0, nb - 1, size=2048), [0, nb - 2]]))
    eidx = torch.from_numpy((kb[:, None] * block + np.arange(block)[None, :]).ravel()).cuda()
    hsrc = [s.index_select(0, eidx).cpu().numpy() for s in src]
    tails = [s[(nb - 1) * block:].cpu().numpy() for s in src]
    codes = [torch.empty((n + 1) // 2, dtype=torch.uint8, device="cuda") for _ in range(P)]
    scales = [torch.empty(nb, dtype=torch.float32, device="cuda") for _ in range(P)]
    out = torch.empty(n, dtype=torch.float32, device="cuda")
    torch.cuda.synchronize()
    for q in range(P):
        zpp.quantize_blockwise_i4(src[q], codes[q], scales[q], block=block)
    zpp.dequant_reduce_i4(codes, scales, n, out, block=block, scale_out=0.125)
    torch.cuda.synchronize()
    del src
    rq = [oracle.quantize_blockwise_i4(h, block) for h in hsrc]
    cidx = torch.from_numpy((kb[:, None] * (block // 2) + np.arange(block // 2)[None, :]).ravel()).cuda()
    sidx = torch.from_numpy(kb).cuda()
    for q in range(P):
        assert_bits_equal(codes[q].index_select(0, cidx).cpu().numpy(), rq[q][0], "codes %d" % q)
        assert_bits_equal(scales[q].index_select(0, sidx).cpu().numpy(), rq[q][1], "scales %d" % q)
    ref = oracle.dequant_reduce_i4([c for c, _ in rq], [s for _, s in rq], kb.size * block, block,
                                   0.125)
    assert_bits_equal(out.index_select(0, eidx).cpu().numpy(), ref, "sampled mean")
    rt = [oracle.quantize_blockwise_i4(t, block) for t in tails]
    lo = (nb - 1) * block
    for q in range(P):
        assert_bits_equal(codes[q][lo // 2:].cpu().numpy(), rt[q][0], "tail codes %d" % q)
    reft = oracle.dequant_reduce_i4([c for c, _ in rt], [s for _, s in rt], n - lo, block, 0.125)
    assert_bits_equal(out[lo:].cpu().numpy(), reft, "tail mean")


# --------------------------------------------------------------------------
# The qgZ receive fused into the partition step
# --------------------------------------------------------------------------
def f32hp(hp):
    return {k: float(np.float32(v)) for k, v in hp.items()}


HP = f32hp(dict(lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1))
HP_LOUD = f32hp(dict(lr=1e-2, beta1=0.8, beta2=0.9, eps=1e-6, weight_decay=0.5))


def receive_state(n, cfg, pad=0, moments=False):
    """Device master / moments / primary (viewed `pad` elements in) for a
    receive step; nonzero moments when `moments`, as after a few steps."""
    p = synth.master_weights(n, cfg)
    m, v = synth.moments(n, cfg) if moments else (np.zeros(n, np.float32),) * 2
    return (to_dev(p, pad=pad), to_dev(m, pad=pad), to_dev(v, pad=pad),
            empty_dev(n, np.uint16, pad=pad, fill=0x5A5A)), (p, m, v)


def run_two_kernels(zpp, quants, n, block, scale_out, state, step, hp, adamw):
    """The reference sequence on the GPU: dequantize-and-reduce into a
    gradient buffer, then the partition step from it."""
    codes = [u8_dev(c) for c, _ in quants]
    scales = [to_dev(s) for _, s in quants]
    g = empty_dev(n, np.float32, fill=-7.0)
    zpp.dequant_reduce_i4(codes, scales, n, g, block=block, scale_out=scale_out)
    p, m, v, b = state
    zpp.adam_partition_step(p, m, v, g, b, step=step, adamw=adamw, **hp)
    torch.cuda.synchronize()
    return to_host(g, np.float32)


def run_receive(zpp, quants, n, block, scale_out, state, step, hp, adamw, pad_codes=0):
    codes = [u8_dev(c, pad=pad_codes) for c, _ in quants]
    scales = [to_dev(s) for _, s in quants]
    p, m, v, b = state
    zpp.qgz_receive_adam_step(p, m, v, codes, scales, b, step=step, adamw=adamw, block=block,
                              scale_out=scale_out, **hp)
    torch.cuda.synchronize()


def host_state(state):
    p, m, v, b = state
    return (to_host(p, np.float32), to_host(m, np.float32), to_host(v, np.float32),
            to_host(b, np.uint16))


# (hyperparameters, moments before the step, step, AdamW or L2): the
# workload's from zero moments at step 1, and exaggerated ones (decay and eps
# visible) from random moments at step 3, as in the partition-step tests
REGIMES = {"workload": (HP, False, 1, True), "loud-adamw": (HP_LOUD, True, 3, True),
           "loud-l2": (HP_LOUD, True, 3, False)}


@pytest.mark.parametrize("P,n,block", [
    (1, 1, 256), (8, 7, 256), (8, 256, 256), (8, 256 * 9 + 81, 256), (3, 65536 + 8, 64),
    (8, 100001, 128), (5, 256 * 33, 1024), (8, 1 << 18, 4096), (64, 256 * 5 + 3, 256),
    (9, 256 * 40, 512), (8, 192 * 37 + 5, 192), (3, 320 * 11 + 7, 320)])
@pytest.mark.parametrize("regime", sorted(REGIMES))
def test_receive_adam_equals_reduce_then_step(zpp, P, n, block, regime):
    """Bit for bit the dequantize-and-reduce followed by the partition step
    (both on the GPU, from the same state), and within the Adam bar of the
    oracle's two functions in sequence."""
    hp, moments, step, adamw = REGIMES[regime]
    quants = oracle_sources(P, n, block, 90 + P + n)
    scale_out = float(np.float32(1.0 / P))
    ref_state, host0 = receive_state(n, 91, moments=moments)
    got_state, _ = receive_state(n, 91, moments=moments)
    g = run_two_kernels(zpp, quants, n, block, scale_out, ref_state, step, hp, adamw)
    run_receive(zpp, quants, n, block, scale_out, got_state, step, hp, adamw)
    got, ref = host_state(got_state), host_state(ref_state)
    for i, name in enumerate(("master", "exp_avg", "exp_avg_sq", "primary")):
        assert_bits_equal(got[i], ref[i], "%s P=%d n=%d block=%d" % (name, P, n, block))
    rg = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], n, block,
                                  scale_out)
    assert_bits_equal(g, rg, "reduced gradient")
    p, m, v = host0
    r = oracle.adam_step(p, m, v, rg, step=step, adamw=adamw, **hp)
    tau_m = first_moment_scale((p, m, v), rg, hp, adamw)
    assert_adam_close(got, r, hp["lr"], "receive step vs oracle", m_tau=tau_m)


@pytest.mark.parametrize("pads", [(1, 0), (0, 1), (3, 1)], ids=["state", "codes", "both"])
def test_receive_adam_misaligned(zpp, pads):
    """Misaligned state or codes take the any-alignment kernel: still the
    two-kernel sequence bit for bit."""
    n, block, P = 256 * 11 + 5, 128, 5
    quants = oracle_sources(P, n, block, 92)
    ref_state, _ = receive_state(n, 93)
    got_state, _ = receive_state(n, 93, pad=pads[0])
    run_two_kernels(zpp, quants, n, block, 0.2, ref_state, 1, HP, True)
    run_receive(zpp, quants, n, block, 0.2, got_state, 1, HP, True, pad_codes=pads[1])
    for a, b in zip(host_state(got_state), host_state(ref_state)):
        assert_bits_equal(a, b, "misaligned %s" % (pads,))


def test_receive_adam_special_scales(zpp):
    """NaN, Inf, zero and subnormal source scales reach the update as the
    reduce forms them."""
    n, block, P = 256 * 8, 256, 4
    quants = oracle_sources(P, n, block, 94)
    quants[1][1][2] = np.nan
    quants[2][1][3] = np.inf
    quants[3][1][4] = 0.0
    quants[0][1][5] = 1e-40
    ref_state, _ = receive_state(n, 95)
    got_state, _ = receive_state(n, 95)
    run_two_kernels(zpp, quants, n, block, 1.0, ref_state, 1, HP, True)
    run_receive(zpp, quants, n, block, 1.0, got_state, 1, HP, True)
    for a, b in zip(host_state(got_state), host_state(ref_state)):
        assert_bits_equal(a, b, "special scales")


def test_fullsize_receive_adam(zpp):
    """The Llama-2-13B partition from 8 int4 sources (arbitrary packed codes
    and scales drawn by the input generator, every nibble from -8 to 7): the
    whole state after the fused receive equals the reduce-then-step sequence
    (compared on the device), and the whole gradient the sequence formed
    equals the oracle's reduction of the same copies."""
    import os
    from concurrent.futures import ThreadPoolExecutor
    wl = WORKLOADS["llama-2-13b"]
    n, block, P = wl.n, wl.block, 8
    nb = (n + block - 1) // block
    hp = f32hp(wl.adam)
    codes = [synth.device_random_packed_i4((n + 1) // 2, wl.cfg_id, rank=q) for q in range(P)]
    scales = [synth.device_random_scales(nb, wl.cfg_id, rank=q, lo=1e-5, hi=2e-4)
              for q in range(P)]
    p0 = synth.device_normal_f32(n, synth.WEIGHT_STD, wl.cfg_id, synth.KIND_MASTER)
    states = []
    for _ in range(2):
        states.append((p0.clone(), torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda"),
                       torch.empty(n, dtype=torch.int16, device="cuda")))
    g = torch.empty(n, dtype=torch.float32, device="cuda")
    zpp.dequant_reduce_i4(codes, scales, n, g, block=block, scale_out=1.0 / P)
    p, m, v, b = states[0]
    zpp.adam_partition_step(p, m, v, g, b, step=1, **hp)
    p, m, v, b = states[1]
    zpp.qgz_receive_adam_step(p, m, v, codes, scales, b, step=1, block=block, scale_out=1.0 / P,
                              **hp)
    torch.cuda.synchronize()
    for a, r, name in zip(states[1], states[0], ("master", "exp_avg", "exp_avg_sq", "primary")):
        assert torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                           r.view(torch.int32) if r.dtype == torch.float32 else r), name
    hc = [c.cpu().numpy() for c in codes]
    hs = [x.cpu().numpy() for x in scales]
    step = -(-n // 64) // block * block
    try:
        k = len(os.sched_getaffinity(0))
    except AttributeError:
        k = os.cpu_count() or 1
    with ThreadPoolExecutor(max(1, min(16, k))) as ex:
        parts = list(ex.map(lambda a: oracle.dequant_reduce_i4(
            [c[a // 2:(a + step) // 2 + 1] for c in hc],
            [x[a // block:-(-(a + step) // block)] for x in hs],
            min(step, n - a), block, float(np.float32(1.0 / P))), range(0, n, step)))
    assert_bits_equal(g.cpu().numpy(), np.concatenate(parts), "whole gradient")


# --------------------------------------------------------------------------
# The whole pass with the receive: step from int4 copies, refresh, quantize
# --------------------------------------------------------------------------
def run_receive_then_refresh_quantize(zpp, quants, n, grad_block, block, scale_out, state,
                                      secondary, step, hp, adamw):
    """The reference sequence on the GPU: the receive step, the refresh of
    the secondary from its primary, the quantization of the primary."""
    p, m, v, b = state
    codes = [u8_dev(c) for c, _ in quants]
    scales = [to_dev(s) for _, s in quants]
    zpp.qgz_receive_adam_step(p, m, v, codes, scales, b, step=step, adamw=adamw,
                              block=grad_block, scale_out=scale_out, **hp)
    sec = empty_dev(n, np.uint16, fill=0x7FC0)
    zpp.refresh_secondary(sec, b)
    qc = empty_dev(n, np.int8, fill=0)
    qs = empty_dev((n + block - 1) // block, np.float32, fill=-1.0)
    zpp.quantize_blockwise_i8(b, qc, qs, block=block)
    torch.cuda.synchronize()
    return host_state(state) + ((to_host(sec, np.uint16) if secondary else None),
                                to_host(qc, np.int8), to_host(qs, np.float32))


def run_receive_pass(zpp, quants, n, grad_block, block, scale_out, state, secondary, step, hp,
                     adamw, pad=0):
    p, m, v, b = state
    codes = [u8_dev(c, pad=pad) for c, _ in quants]
    scales = [to_dev(s) for _, s in quants]
    sec = empty_dev(n, np.uint16, pad=pad, fill=0x7FC0) if secondary else None
    qc = empty_dev(n, np.int8, pad=pad, fill=0)
    qs = empty_dev((n + block - 1) // block, np.float32, fill=-1.0)
    zpp.qgz_receive_step_refresh_quantize(p, m, v, codes, scales, b, sec, qc, qs, step=step,
                                          adamw=adamw, grad_block=grad_block, block=block,
                                          scale_out=scale_out, **hp)
    torch.cuda.synchronize()
    return host_state(state) + ((to_host(sec, np.uint16) if secondary else None),
                                to_host(qc, np.int8), to_host(qs, np.float32))


@pytest.mark.parametrize("P,n,grad_block,block,secondary", [
    (8, 256 * 40, 256, 256, True), (8, 256 * 9 + 81, 256, 256, True),
    (3, 65536 + 8, 64, 1024, False), (5, 100001, 512, 128, True), (1, 7, 256, 64, True),
    (64, 256 * 5 + 3, 256, 4096, True), (8, 1 << 18, 4096, 256, False),
    (8, 192 * 37 + 5, 192, 320, True), (3, 320 * 11 + 7, 320, 192, False),
    (8, 2112 * 5 + 17, 256, 2112, True)])
@pytest.mark.parametrize("regime", sorted(REGIMES))
def test_receive_pass_equals_three_calls(zpp, P, n, grad_block, block, secondary, regime):
    """Bit for bit the receive step, then the refresh and the quantization of
    its primary (all on the GPU, from the same state)."""
    hp, moments, step, adamw = REGIMES[regime]
    quants = oracle_sources(P, n, grad_block, 96 + P + n)
    scale_out = float(np.float32(1.0 / P))
    ref_state, _ = receive_state(n, 97, moments=moments)
    got_state, _ = receive_state(n, 97, moments=moments)
    ref = run_receive_then_refresh_quantize(zpp, quants, n, grad_block, block, scale_out,
                                            ref_state, secondary, step, hp, adamw)
    got = run_receive_pass(zpp, quants, n, grad_block, block, scale_out, got_state, secondary,
                           step, hp, adamw)
    names = ("master", "exp_avg", "exp_avg_sq", "primary", "secondary", "codes", "scales")
    for a, b, name in zip(got, ref, names):
        if a is None:
            continue
        assert_bits_equal(a, b, "%s P=%d n=%d blocks %d/%d" % (name, P, n, grad_block, block))


@pytest.mark.parametrize("pad", [1, 3])
def test_receive_pass_misaligned(zpp, pad):
    """Misaligned arrays take the three scalar kernels: the same results."""
    n, grad_block, block, P = 256 * 11 + 5, 128, 256, 5
    quants = oracle_sources(P, n, grad_block, 98)
    ref_state, _ = receive_state(n, 99)
    got_state, _ = receive_state(n, 99, pad=pad)
    ref = run_receive_then_refresh_quantize(zpp, quants, n, grad_block, block, 0.2, ref_state,
                                            True, 1, HP, True)
    got = run_receive_pass(zpp, quants, n, grad_block, block, 0.2, got_state, True, 1, HP, True,
                           pad=pad)
    for a, b in zip(got, ref):
        assert_bits_equal(a, b, "misaligned pad=%d" % pad)


def test_receive_pass_special_scales(zpp):
    """NaN, Inf, zero and subnormal source scales through the single pass:
    the blocks they poison quantize as the separate quantizer quantizes them
    (NaN scale, zero codes), everything else bit for bit as the three calls."""
    n, block, P = 256 * 8 + 40, 256, 4
    quants = oracle_sources(P, n, block, 102)
    quants[1][1][2] = np.nan
    quants[2][1][3] = np.inf
    quants[3][1][4] = 0.0
    quants[0][1][5] = 1e-40
    quants[2][1][8] = np.nan  # the partial last block
    ref_state, _ = receive_state(n, 103)
    got_state, _ = receive_state(n, 103)
    ref = run_receive_then_refresh_quantize(zpp, quants, n, block, block, 1.0, ref_state, True,
                                            1, HP, True)
    got = run_receive_pass(zpp, quants, n, block, block, 1.0, got_state, True, 1, HP, True)
    names = ("master", "exp_avg", "exp_avg_sq", "primary", "secondary", "codes", "scales")
    for a, b, name in zip(got, ref, names):
        assert_bits_equal(a, b, "special scales, " + name)
    scales = got[6].view(np.uint32)
    assert scales[2] == 0x7FC00000 and scales[8] == 0x7FC00000, "poisoned blocks keep NaN scales"
    assert not got[5][2 * 256:3 * 256].any(), "a NaN block's codes are zero"


def test_fullsize_receive_pass(zpp):
    """The Llama-2-13B partition from 8 int4 sources: the single pass equals
    the receive step, the refresh and the quantization, compared whole on the
    device."""
    wl = WORKLOADS["llama-2-13b"]
    n, B, P = wl.n, wl.block, 8
    nb = (n + B - 1) // B
    hp = f32hp(wl.adam)
    codes = [torch.empty((n + 1) // 2, dtype=torch.uint8, device="cuda") for _ in range(P)]
    scales = [torch.empty(nb, dtype=torch.float32, device="cuda") for _ in range(P)]
    for q in range(P):
        src = synth.device_normal_f32(n, synth.GRAD_STD, wl.cfg_id, synth.KIND_GRAD, rank=q)
        zpp.quantize_blockwise_i4(src, codes[q], scales[q], block=B)
        torch.cuda.synchronize()
        del src
    p0 = synth.device_normal_f32(n, synth.WEIGHT_STD, wl.cfg_id, synth.KIND_MASTER)
    outs = []
    for single in (False, True):
        p, m, v = p0.clone(), torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
        prim = torch.empty(n, dtype=torch.int16, device="cuda")
        sec = torch.empty(n, dtype=torch.int16, device="cuda")
        qc = torch.empty(n, dtype=torch.int8, device="cuda")
        qs = torch.empty(nb, dtype=torch.float32, device="cuda")
        if single:
            zpp.qgz_receive_step_refresh_quantize(p, m, v, codes, scales, prim, sec, qc, qs,
                                                  step=1, scale_out=1.0 / P, **hp)
        else:
            zpp.qgz_receive_adam_step(p, m, v, codes, scales, prim, step=1, scale_out=1.0 / P,
                                      **hp)
            zpp.refresh_secondary(sec, prim)
            zpp.quantize_blockwise_i8(prim, qc, qs)
        torch.cuda.synchronize()
        outs.append([p.view(torch.int32), m.view(torch.int32), v.view(torch.int32), prim, sec,
                     qc, qs.view(torch.int32)])
    for a, b, name in zip(outs[1], outs[0], ("master", "exp_avg", "exp_avg_sq", "primary",
                                             "secondary", "codes", "scales")):
        assert torch.equal(a, b), name


# ===========================================================================
# The interleaved receive buffer: the P int4 copies in one buffer, block by
# block (layout in include/zpp.h)
# ===========================================================================
def interleave(quants, n, block):
    """Lay the P separate (codes, scales) out as one interleaved receive
    buffer: block k holds each source's block/2 code bytes side by side, and
    source q's scale of block k is scale k P + q."""
    P = len(quants)
    nb = -(-n // block)
    half = block // 2
    codes = np.zeros((nb, P, half), np.uint8)
    scales = np.zeros((nb, P), np.float32)
    for q, (c, s) in enumerate(quants):
        padded = np.zeros(nb * half, np.uint8)
        padded[:c.size] = c
        codes[:, q, :] = padded.reshape(nb, half)
        scales[:, q] = s
    return codes.ravel(), scales.ravel()


def deinterleave(codes, scales, n, block, P):
    nb = -(-n // block)
    half = block // 2
    c = codes[:nb * P * half].reshape(nb, P, half)
    s = scales[:nb * P].reshape(nb, P)
    return [(c[:, q, :].ravel()[:(n + 1) // 2].copy(), s[:, q].copy()) for q in range(P)]


def zeros_u8(n):
    return torch.zeros(n, dtype=torch.uint8, device="cuda")


@pytest.mark.parametrize("P,n,block", [(1, 7, 256), (3, 256 * 9 + 81, 64), (8, 100001, 256),
                                       (8, 65536 + 8, 1024), (64, 256 * 5 + 3, 128),
                                       (5, 4096 * 3 + 500, 4096), (8, 192 * 9 + 81, 192),
                                       (3, 320 * 5 + 3, 320)])
@pytest.mark.parametrize("pad", [0, 1], ids=["vector", "scalar"])
def test_quantize_i4_interleaved_equals_plain(zpp, P, n, block, pad):
    """Each source quantized into its slots of one interleaved buffer: taken
    back out, every source's codes and scales are the oracle's, bit for bit."""
    srcs = [grads(n, 150 + P, q, scale=1.0 + q) for q in range(P)]
    nc, ns = zpp.interleaved_sizes(n, block, P)
    codes = zeros_u8(nc)
    scales = empty_dev(ns, np.float32, fill=-1.0)
    for q, x in enumerate(srcs):
        zpp.quantize_blockwise_i4_interleaved(to_dev(x, pad=pad), codes, scales, source=q,
                                              num_src=P, block=block)
    torch.cuda.synchronize()
    got = deinterleave(codes.cpu().numpy(), to_host(scales, np.float32), n, block, P)
    for q, x in enumerate(srcs):
        rc, rs = oracle.quantize_blockwise_i4(x, block)
        assert_bits_equal(got[q][0], rc, "codes of source %d" % q)
        assert_bits_equal(got[q][1], rs, "scales of source %d" % q)


def run_receive_il(zpp, quants, n, block, scale_out, state, step, hp, adamw, pad_codes=0):
    ic, isc = interleave(quants, n, block)
    p, m, v, b = state
    zpp.qgz_receive_adam_step_interleaved(p, m, v, u8_dev(ic, pad=pad_codes), to_dev(isc),
                                          len(quants), b, step=step, adamw=adamw, block=block,
                                          scale_out=scale_out, **hp)
    torch.cuda.synchronize()


@pytest.mark.parametrize("P,n,block", [
    (1, 1, 256), (8, 7, 256), (8, 256 * 9 + 81, 256), (3, 65536 + 8, 64), (8, 100001, 128),
    (5, 256 * 33, 1024), (8, 1 << 18, 4096), (64, 256 * 5 + 3, 256), (9, 256 * 40, 512),
    (16, 256 * 17 + 100, 64), (8, 192 * 9 + 81, 192), (3, 320 * 11 + 7, 320)])
@pytest.mark.parametrize("regime", sorted(REGIMES))
def test_receive_interleaved_equals_separate(zpp, P, n, block, regime):
    """The receive step from one interleaved buffer leaves the same bits as
    from the P separate arrays (same state, same sources)."""
    hp, moments, step, adamw = REGIMES[regime]
    quants = oracle_sources(P, n, block, 160 + P + n)
    scale_out = float(np.float32(1.0 / P))
    ref_state, _ = receive_state(n, 161, moments=moments)
    got_state, _ = receive_state(n, 161, moments=moments)
    run_receive(zpp, quants, n, block, scale_out, ref_state, step, hp, adamw)
    run_receive_il(zpp, quants, n, block, scale_out, got_state, step, hp, adamw)
    for a, b, name in zip(host_state(got_state), host_state(ref_state),
                          ("master", "exp_avg", "exp_avg_sq", "primary")):
        assert_bits_equal(a, b, "%s P=%d n=%d block %d" % (name, P, n, block))


@pytest.mark.parametrize("pads", [(1, 0), (0, 1), (0, 3), (0, 2)],
                         ids=["state", "codes-odd", "codes-odd-3", "codes-2"])
def test_receive_interleaved_misaligned(zpp, pads):
    """Misaligned state, or interleaved codes at an odd address, take the
    any-alignment kernel; codes at a 2-byte address keep the vector kernel:
    the same bits either way."""
    n, block, P = 256 * 11 + 5, 128, 5
    quants = oracle_sources(P, n, block, 162)
    ref_state, _ = receive_state(n, 163)
    got_state, _ = receive_state(n, 163, pad=pads[0])
    run_receive(zpp, quants, n, block, 0.2, ref_state, 1, HP, True)
    run_receive_il(zpp, quants, n, block, 0.2, got_state, 1, HP, True, pad_codes=pads[1])
    for a, b in zip(host_state(got_state), host_state(ref_state)):
        assert_bits_equal(a, b, "misaligned %s" % (pads,))


def test_receive_interleaved_vs_oracle(zpp):
    """The interleaved receive step against the oracle's dequantize-and-reduce
    of the same sources followed by its Adam step."""
    n, block, P = 256 * 21 + 17, 256, 8
    hp = HP_LOUD
    quants = oracle_sources(P, n, block, 164)
    state, (p, m, v) = receive_state(n, 165, moments=True)
    run_receive_il(zpp, quants, n, block, float(np.float32(1.0 / P)), state, 3, hp, True)
    g = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], n, block,
                                 float(np.float32(1.0 / P)))
    ref = oracle.adam_step(p, m, v, g, step=3, **hp)
    assert_adam_close(host_state(state), ref, hp["lr"], "interleaved receive", prev=(p, m, v),
                      g=g, hp=hp)


def run_receive_pass_il(zpp, quants, n, grad_block, block, scale_out, state, secondary, step,
                        hp, adamw, pad=0):
    p, m, v, b = state
    ic, isc = interleave(quants, n, grad_block)
    sec = empty_dev(n, np.uint16, pad=pad, fill=0x7FC0) if secondary else None
    qc = empty_dev(n, np.int8, pad=pad, fill=0)
    qs = empty_dev((n + block - 1) // block, np.float32, fill=-1.0)
    zpp.qgz_receive_step_refresh_quantize_interleaved(
        p, m, v, u8_dev(ic), to_dev(isc), len(quants), b, sec, qc, qs, step=step, adamw=adamw,
        grad_block=grad_block, block=block, scale_out=scale_out, **hp)
    torch.cuda.synchronize()
    return host_state(state) + ((to_host(sec, np.uint16) if secondary else None),
                                to_host(qc, np.int8), to_host(qs, np.float32))


@pytest.mark.parametrize("P,n,grad_block,block,secondary", [
    (8, 256 * 40, 256, 256, True), (8, 256 * 9 + 81, 256, 256, True),
    (3, 65536 + 8, 64, 1024, False), (5, 100001, 512, 128, True), (1, 7, 256, 64, True),
    (64, 256 * 5 + 3, 256, 4096, True), (8, 1 << 18, 4096, 256, False),
    (16, 256 * 17 + 100, 128, 512, True), (8, 192 * 37 + 5, 192, 320, True),
    (13, 256 * 9 + 81, 256, 256, True), (8, 2112 * 5 + 17, 256, 2112, True)])
@pytest.mark.parametrize("regime", sorted(REGIMES))
def test_receive_pass_interleaved_equals_separate(zpp, P, n, grad_block, block, secondary,
                                                  regime):
    """The single pass from one interleaved buffer: the same bits as from the
    P separate arrays."""
    hp, moments, step, adamw = REGIMES[regime]
    quants = oracle_sources(P, n, grad_block, 166 + P + n)
    scale_out = float(np.float32(1.0 / P))
    ref_state, _ = receive_state(n, 167, moments=moments)
    got_state, _ = receive_state(n, 167, moments=moments)
    ref = run_receive_pass(zpp, quants, n, grad_block, block, scale_out, ref_state, secondary,
                           step, hp, adamw)
    got = run_receive_pass_il(zpp, quants, n, grad_block, block, scale_out, got_state,
                              secondary, step, hp, adamw)
    names = ("master", "exp_avg", "exp_avg_sq", "primary", "secondary", "codes", "scales")
    for a, b, name in zip(got, ref, names):
        if a is None:
            continue
        assert_bits_equal(a, b, "%s P=%d n=%d blocks %d/%d" % (name, P, n, grad_block, block))


def test_fullsize_receive_interleaved(zpp):
    """The Llama-2-13B partition from 8 int4 sources, each quantized on the
    device into separate arrays and into one interleaved buffer: the receive
    step and the single pass leave the same bits either way (compared whole
    on the device)."""
    wl = WORKLOADS["llama-2-13b"]
    n, B, P = wl.n, wl.block, 8
    nb = (n + B - 1) // B
    hp = f32hp(wl.adam)
    codes = [torch.empty((n + 1) // 2, dtype=torch.uint8, device="cuda") for _ in range(P)]
    scales = [torch.empty(nb, dtype=torch.float32, device="cuda") for _ in range(P)]
    nc, ns = zpp.interleaved_sizes(n, B, P)
    ic = torch.zeros(nc, dtype=torch.uint8, device="cuda")
    isc = torch.zeros(ns, dtype=torch.float32, device="cuda")
    for q in range(P):
        src = synth.device_normal_f32(n, synth.GRAD_STD, wl.cfg_id, synth.KIND_GRAD, rank=q)
        zpp.quantize_blockwise_i4(src, codes[q], scales[q], block=B)
        zpp.quantize_blockwise_i4_interleaved(src, ic, isc, source=q, num_src=P, block=B)
        torch.cuda.synchronize()
        del src
    p0 = synth.device_normal_f32(n, synth.WEIGHT_STD, wl.cfg_id, synth.KIND_MASTER)
    for single in (False, True):
        outs = []
        for il in (False, True):
            p, m, v = p0.clone(), torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
            prim = torch.empty(n, dtype=torch.int16, device="cuda")
            sec = torch.empty(n, dtype=torch.int16, device="cuda")
            qc = torch.empty(n, dtype=torch.int8, device="cuda")
            qs = torch.empty(nb, dtype=torch.float32, device="cuda")
            if single and il:
                zpp.qgz_receive_step_refresh_quantize_interleaved(
                    p, m, v, ic, isc, P, prim, sec, qc, qs, step=1, scale_out=1.0 / P, **hp)
            elif single:
                zpp.qgz_receive_step_refresh_quantize(p, m, v, codes, scales, prim, sec, qc, qs,
                                                      step=1, scale_out=1.0 / P, **hp)
            elif il:
                zpp.qgz_receive_adam_step_interleaved(p, m, v, ic, isc, P, prim, step=1,
                                                      scale_out=1.0 / P, **hp)
            else:
                zpp.qgz_receive_adam_step(p, m, v, codes, scales, prim, step=1,
                                          scale_out=1.0 / P, **hp)
            torch.cuda.synchronize()
            outs.append([p, m, v, prim] + ([sec, qc, qs] if single else []))
        for a, b in zip(*outs):
            assert torch.equal(a, b), "interleaved %s differs" % ("pass" if single else "step")
        del outs
        torch.cuda.empty_cache()


def run_reduce_il(zpp, quants, n, block, scale_out, pad_out=0, pad_codes=0):
    ic, isc = interleave(quants, n, block)
    out = empty_dev(n, np.float32, pad=pad_out, fill=-7.0)
    zpp.dequant_reduce_i4_interleaved(u8_dev(ic, pad=pad_codes), to_dev(isc), len(quants), n,
                                      out, block=block, scale_out=scale_out)
    torch.cuda.synchronize()
    return to_host(out, np.float32)


@pytest.mark.parametrize("P,n,block", [
    (1, 1, 256), (2, 7, 64), (8, 9, 256), (3, 256 * 5 + 3, 128), (8, 65536 + 8, 256),
    (8, 100001, 1024), (64, 256 * 5 + 3, 256), (5, 4096 * 3 + 500, 4096), (16, 512 * 9, 64),
    (8, 320 * 9 + 81, 320), (3, 192 * 5 + 3, 192), (13, 256 * 7 + 5, 256)])
def test_dequant_reduce_interleaved_vs_oracle(zpp, P, n, block):
    """The dequant-reduce from one interleaved receive buffer against the
    oracle's reduction of the same P copies (separate arrays), bit for bit."""
    quants = oracle_sources(P, n, block, 170 + n)
    for scale_out in (1.0, float(np.float32(1.0 / P))):
        got = run_reduce_il(zpp, quants, n, block, scale_out)
        ref = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], n, block,
                                       scale_out)
        assert_bits_equal(got, ref, "P=%d n=%d block %d scale_out=%g" % (P, n, block, scale_out))


@pytest.mark.parametrize("pads", [(1, 0), (0, 1), (0, 2)], ids=["out", "codes-odd", "codes-2"])
def test_dequant_reduce_interleaved_misaligned(zpp, pads):
    """A misaligned output or codes at an odd address take the any-alignment
    kernel; codes at a 2-byte address keep the vector kernel: the oracle's
    bits either way."""
    n, block, P = 256 * 11 + 5, 128, 5
    quants = oracle_sources(P, n, block, 171)
    got = run_reduce_il(zpp, quants, n, block, 0.2, *pads)
    ref = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], n, block,
                                   float(np.float32(0.2)))
    assert_bits_equal(got, ref, "misaligned %s" % (pads,))


def test_dequant_reduce_interleaved_special_scales(zpp):
    """NaN, Inf, zero and subnormal source scales reach the output as the
    oracle's reduction has them."""
    n, block, P = 256 * 8, 256, 4
    quants = oracle_sources(P, n, block, 172)
    quants[1][1][2] = np.nan
    quants[2][1][3] = np.inf
    quants[3][1][4] = 0.0
    quants[0][1][5] = 1e-40
    got = run_reduce_il(zpp, quants, n, block, 1.0)
    ref = oracle.dequant_reduce_i4([c for c, _ in quants], [s for _, s in quants], n, block, 1.0)
    assert_bits_equal(got, ref, "special scales")


def test_fullsize_reduce_interleaved(zpp):
    """The Llama-2-13B partition from 8 int4 sources quantized on the device
    into separate arrays and into one interleaved buffer: the two reductions
    are equal bit for bit, and sampled blocks (the partial last one among
    them) equal the oracle's quantization and reduction of the same sources."""
    wl = WORKLOADS["llama-2-13b"]
    n, B, P = wl.n, wl.block, 8
    nb = (n + B - 1) // B
    g = np.random.default_rng(173)
    kb = np.unique(np.concatenate([g.integers(0, nb - 1, size=512), [0, nb - 2]]))
    eidx = torch.from_numpy((kb[:, None] * B + np.arange(B)[None, :]).ravel()).cuda()
    lo = (nb - 1) * B
    codes = [torch.empty((n + 1) // 2, dtype=torch.uint8, device="cuda") for _ in range(P)]
    scales = [torch.empty(nb, dtype=torch.float32, device="cuda") for _ in range(P)]
    nc, ns = zpp.interleaved_sizes(n, B, P)
    ic = torch.zeros(nc, dtype=torch.uint8, device="cuda")
    isc = torch.zeros(ns, dtype=torch.float32, device="cuda")
    hsrc, tails = [], []
    for q in range(P):
        src = synth.device_normal_f32(n, synth.GRAD_STD, wl.cfg_id, synth.KIND_GRAD, rank=q)
        hsrc.append(src.index_select(0, eidx).cpu().numpy())
        tails.append(src[lo:].cpu().numpy())
        zpp.quantize_blockwise_i4(src, codes[q], scales[q], block=B)
        zpp.quantize_blockwise_i4_interleaved(src, ic, isc, source=q, num_src=P, block=B)
        torch.cuda.synchronize()
        del src
    outs = []
    for il in (False, True):
        out = torch.empty(n, dtype=torch.float32, device="cuda")
        if il:
            zpp.dequant_reduce_i4_interleaved(ic, isc, P, n, out, block=B, scale_out=0.125)
        else:
            zpp.dequant_reduce_i4(codes, scales, n, out, block=B, scale_out=0.125)
        torch.cuda.synchronize()
        outs.append(out)
    assert torch.equal(outs[0], outs[1])
    rq = [oracle.quantize_blockwise_i4(h, B) for h in hsrc]
    ref = oracle.dequant_reduce_i4([c for c, _ in rq], [s for _, s in rq], kb.size * B, B, 0.125)
    assert_bits_equal(outs[1].index_select(0, eidx).cpu().numpy(), ref, "sampled mean")
    rt = [oracle.quantize_blockwise_i4(t, B) for t in tails]
    reft = oracle.dequant_reduce_i4([c for c, _ in rt], [s for _, s in rt], n - lo, B, 0.125)
    assert_bits_equal(outs[1][lo:].cpu().numpy(), reft, "tail mean")
    del outs, codes, scales, ic, isc
    torch.cuda.empty_cache()
