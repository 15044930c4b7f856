"""GPU parity: every kernel of the partition path, called through the C ABI,
against the CPU oracle on identical seeded inputs.

Sizes span several tiles with ragged tails; misaligned views drive the
scalar kernels; special values cover the degenerate cases of the method.
Full-size cases at the Llama-2-13B shapes live in test_gpu_fullsize.py.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2407_01614_amd import synth
from paper_2407_01614_amd.workloads import WORKLOADS, secondary_elems
from parity import (MomentTolerance, assert_adam_close, assert_bits_equal, empty_dev, to_dev,
                    to_host)

pytestmark = pytest.mark.gpu

TINY = WORKLOADS["tiny"]
HP_TINY = dict(lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
HP_LOUD = dict(lr=1e-2, beta1=0.8, beta2=0.9, eps=1e-6, weight_decay=0.5)


@pytest.fixture(scope="module")
def zpp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2407_01614_amd import zpp as mod
    return mod


def f32hp(hp):
    return {k: float(np.float32(v)) for k, v in hp.items()}


# ===========================================================================
# Adam partition step
# ===========================================================================
def run_adam_gpu(zpp, p, m, v, g, hp, step, adamw=True, pad=0):
    tp, tm, tv, tg = (to_dev(x, pad=pad) for x in (p, m, v, g))
    out = empty_dev(p.size, np.uint16, pad=pad, fill=0x5555)
    zpp.adam_partition_step(tp, tm, tv, tg, out, step=step, adamw=adamw, **hp)
    torch.cuda.synchronize()
    return (to_host(tp, np.float32), to_host(tm, np.float32), to_host(tv, np.float32),
            to_host(out, np.uint16))


def test_adam_tiny_four_ranks(zpp):
    """The Tiny workload: 4 simulated ranks, each a 1,048,576-element
    partition, step 1 from zero moments."""
    hp = f32hp(HP_TINY)
    n = TINY.n
    for rank in range(TINY.world):
        p = synth.master_weights(n, TINY.cfg_id, rank)
        g = synth.gradients(n, TINY.cfg_id, rank)
        z = np.zeros(n, np.float32)
        got = run_adam_gpu(zpp, p, z, z, g, hp, 1)
        ref = oracle.adam_step(p, z, z, g, step=1, **hp)
        assert_adam_close(got, ref, hp["lr"], "rank %d" % rank)


@pytest.mark.parametrize("adamw", [True, False])
@pytest.mark.parametrize("hp", [HP_TINY, HP_LOUD], ids=["tiny-hp", "loud-hp"])
def test_adam_multistep(zpp, adamw, hp):
    hp = f32hp(hp)
    n = 3 * 2048 + 77
    p = synth.master_weights(n, 40)
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    rp, rm, rv = p, m, v
    tp, tm, tv = (to_dev(x) for x in (p, m, v))
    out = empty_dev(n, np.uint16)
    mt = MomentTolerance()
    gp = p
    for t in range(1, 8):
        g = synth.gradients(n, 40, it=t) * np.float32(5.0)
        zpp.adam_partition_step(tp, tm, tv, to_dev(g), out, step=t, adamw=adamw, **hp)
        # in the L2 form the masters' difference enters the first moment
        tau_m = mt.step((rp, rm, rv), g, hp, adamw,
                        p_diff=gp.astype(np.float64) - rp.astype(np.float64))
        rp, rm, rv, rb = oracle.adam_step(rp, rm, rv, g, step=t, adamw=adamw, **hp)
        torch.cuda.synchronize()
        got = (to_host(tp, np.float32), to_host(tm, np.float32), to_host(tv, np.float32),
               to_host(out, np.uint16))
        assert_adam_close(got, (rp, rm, rv, rb), hp["lr"], "step %d" % t, m_tau=tau_m)
        gp = got[0]


@pytest.mark.parametrize("n", [1, 3, 4, 5, 1023, 2047, 2048, 2049, 3 * 2048 + 7, 100003])
@pytest.mark.parametrize("pad", [0, 1], ids=["vector", "scalar"])
def test_adam_ragged(zpp, n, pad):
    hp = f32hp(HP_LOUD)
    p = synth.master_weights(n, 41, n)
    g = synth.gradients(n, 41, n)
    m, v = synth.moments(n, 41, n)
    got = run_adam_gpu(zpp, p, m, v, g, hp, 3, pad=pad)
    ref = oracle.adam_step(p, m, v, g, step=3, **hp)
    assert_adam_close(got, ref, hp["lr"], "n=%d pad=%d" % (n, pad), prev=(p, m, v), g=g, hp=hp)


def test_adam_nonfinite_and_zero_grads(zpp):
    hp = f32hp(HP_TINY)
    n = 4096
    p = synth.master_weights(n, 42)
    g = synth.gradients(n, 42)
    g[::7] = 0.0
    g[5] = np.inf
    g[900] = -np.inf
    g[2049] = np.nan
    p[3000] = np.float32(3.0e38)  # decays, stays finite
    z = np.zeros(n, np.float32)
    got = run_adam_gpu(zpp, p, z, z, g, hp, 1)
    ref = oracle.adam_step(p, z, z, g, step=1, **hp)
    assert_adam_close(got, ref, hp["lr"])
    assert np.isnan(got[0][[5, 900, 2049]]).all()


def test_adam_large_step_count(zpp):
    hp = f32hp(HP_TINY)
    n = 65536 + 3
    p = synth.master_weights(n, 43)
    g = synth.gradients(n, 43)
    m, v = synth.moments(n, 43)
    got = run_adam_gpu(zpp, p, m, v, g, hp, 123456)
    ref = oracle.adam_step(p, m, v, g, step=123456, **hp)
    assert_adam_close(got, ref, hp["lr"], prev=(p, m, v), g=g, hp=hp)


DEGENERATE = {
    "lr=0": dict(lr=0.0, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1),
    "wd=0": dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.0),
    "beta1=0": dict(lr=1e-3, beta1=0.0, beta2=0.95, eps=1e-8, weight_decay=0.1),
    "beta2=0": dict(lr=1e-3, beta1=0.9, beta2=0.0, eps=1e-8, weight_decay=0.1),
    "betas=0": dict(lr=1e-3, beta1=0.0, beta2=0.0, eps=1e-8, weight_decay=0.1),
    "eps=0": dict(lr=1e-3, beta1=0.9, beta2=0.95, eps=0.0, weight_decay=0.1),
}


@pytest.mark.parametrize("adamw", [True, False], ids=["adamw", "l2"])
@pytest.mark.parametrize("case", sorted(DEGENERATE))
def test_adam_degenerate_hyperparameters(zpp, case, adamw):
    """Hyperparameters at the edges the method allows, from a mid-training
    state (step 3, nonzero moments): a zero learning rate leaves the master
    bit for bit; zero decay, betas of 0 (no momentum: m = g, v = g^2) and a
    zero eps all match the oracle."""
    hp = f32hp(DEGENERATE[case])
    n = 256 * 37 + 11
    p = synth.master_weights(n, 44)
    g = synth.gradients(n, 44)
    m, v = synth.moments(n, 44)
    got = run_adam_gpu(zpp, p, m, v, g, hp, 3, adamw=adamw)
    ref = oracle.adam_step(p, m, v, g, step=3, adamw=adamw, **hp)
    assert_adam_close(got, ref, hp["lr"], case, prev=(p, m, v), g=g, hp=hp, adamw=adamw)
    if hp["lr"] == 0.0:
        assert_bits_equal(got[0], p, "master with lr = 0")
        assert_bits_equal(got[3], ref[3], "primary with lr = 0")


def test_adam_checkpoint_resume_is_bitwise(zpp):
    """k steps, save the state to the host, reload it into fresh buffers and
    take one more step: bit-identical to k+1 uninterrupted steps."""
    hp = f32hp(HP_TINY)
    n = 50000
    p = synth.master_weights(n, 44)
    tp, tm, tv = to_dev(p), torch.zeros(n, device="cuda"), torch.zeros(n, device="cuda")
    out = empty_dev(n, np.uint16)
    grads = [to_dev(synth.gradients(n, 44, it=t)) for t in range(1, 6)]
    for t in range(1, 5):
        zpp.adam_partition_step(tp, tm, tv, grads[t - 1], out, step=t, **hp)
    torch.cuda.synchronize()
    saved = [x.cpu().clone() for x in (tp, tm, tv)]
    zpp.adam_partition_step(tp, tm, tv, grads[4], out, step=5, **hp)
    rp, rm, rv = (x.cuda() for x in saved)
    out2 = empty_dev(n, np.uint16)
    zpp.adam_partition_step(rp, rm, rv, grads[4], out2, step=5, **hp)
    torch.cuda.synchronize()
    for a, b in ((tp, rp), (tm, rm), (tv, rv), (out, out2)):
        assert torch.equal(a.view(torch.int32) if a.dtype == torch.float32 else a,
                           b.view(torch.int32) if b.dtype == torch.float32 else b)


# ===========================================================================
# Secondary refresh
# ===========================================================================
@pytest.mark.parametrize("count", [0, 1, 7, 8, 9, 8191, 8192, 8193, 2 * 8192 * 4 + 5, 2097152])
@pytest.mark.parametrize("pad", [0, 1], ids=["vector", "scalar"])
def test_refresh_bitwise(zpp, count, pad):
    src = synth.random_bits16(count, 50, count)
    tsrc = to_dev(src, pad=pad)
    dst = empty_dev(count, np.uint16, pad=pad, fill=0x7FC0)
    zpp.refresh_secondary(dst, tsrc)
    torch.cuda.synchronize()
    assert_bits_equal(to_host(dst, np.uint16), oracle.refresh(src), "refresh")


def test_refresh_leaves_bytes_past_count(zpp):
    src = synth.random_bits16(10000, 51)
    dst = empty_dev(10000, np.uint16, fill=0x1234)
    zpp.refresh_secondary(dst, to_dev(src), 9001)
    torch.cuda.synchronize()
    h = to_host(dst, np.uint16)
    assert_bits_equal(h[:9001], src[:9001])
    assert np.all(h[9001:] == 0x1234)


# ===========================================================================
# Quantization
# ===========================================================================
def run_quant_gpu(zpp, x, block, pad_src=0, pad_codes=0):
    tx = to_dev(x, pad=pad_src)
    codes = empty_dev(x.size, np.int8, pad=pad_codes, fill=99)
    nb = (x.size + block - 1) // block
    scales = empty_dev(nb, np.float32, fill=-1.0)
    zpp.quantize_blockwise_i8(tx, codes, scales, block=block)
    torch.cuda.synchronize()
    return to_host(codes, np.int8), to_host(scales, np.float32)


def assert_quant_equal(got, ref, what):
    assert_bits_equal(got[0], ref[0], what + " codes")
    assert_bits_equal(got[1], ref[1], what + " scales")


def test_quant_tiny_secondary_shards(zpp):
    s = TINY.shard_elems
    for j in range(TINY.secondary_world):
        x = synth.bf16_weights(s, TINY.cfg_id, j)
        assert_quant_equal(run_quant_gpu(zpp, x, 256), oracle.quantize_blockwise_i8(x, 256),
                           "shard %d" % j)


@pytest.mark.parametrize("block", [64, 128, 192, 256, 320, 448, 512, 960, 1024, 1088, 2048, 2112,
                                   4032, 4096])
@pytest.mark.parametrize("n", [1, 7, 8, 63, 255, 256, 257, 256 * 5 + 80, 100000, 1 << 17])
def test_quant_blocks_and_ragged(zpp, block, n):
    x = synth.bf16_weights(n, 52, n + block)
    assert_quant_equal(run_quant_gpu(zpp, x, block), oracle.quantize_blockwise_i8(x, block),
                       "n=%d block=%d" % (n, block))


@pytest.mark.parametrize("pads", [(1, 0), (0, 1), (8, 3)], ids=["src", "codes", "both"])
def test_quant_misaligned_scalar_path(zpp, pads):
    n = 256 * 37 + 80
    x = synth.bf16_weights(n, 53)
    assert_quant_equal(run_quant_gpu(zpp, x, 256, *pads), oracle.quantize_blockwise_i8(x, 256),
                       "pads=%s" % (pads,))


def special_blocks(block):
    rng = np.random.default_rng(77)
    parts = []
    base = lambda: (rng.standard_normal(block) * 0.02).astype(np.float32)
    parts.append(np.zeros(block, np.float32))                       # zero block
    b = base(); b[3] = np.inf; parts.append(b)                       # +inf
    b = base(); b[block - 1] = -np.inf; parts.append(b)              # -inf
    b = base(); b[0] = np.nan; parts.append(b)                       # NaN
    for e in (-133, -126, -120, -101, -100, -99, -60, 0, 60, 120):   # tiny .. huge blocks
        q = rng.integers(-127, 128, size=block).astype(np.float64)
        q[rng.integers(0, block)] = 127
        parts.append((q * 2.0 ** e).astype(np.float32))
    b = base(); b[:block // 2] = 0.0; parts.append(b)                # half zeros
    b = np.full(block, -0.0, np.float32); parts.append(b)            # negative zeros
    b = np.array([0.5, 1.5, 2.5, -2.5, 127.0] + [0.0] * (block - 5), np.float32)
    parts.append(b)                                                  # ties to even
    b = (rng.standard_normal(block) * 1e-39).astype(np.float32); parts.append(b)  # subnormal
    x = np.concatenate(parts)
    bits = (x.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    bits[block * 3 + 7] = 0x7F81  # signalling-looking NaN payload
    return bits


@pytest.mark.parametrize("block", [64, 192, 256, 4032, 4096])
@pytest.mark.parametrize("pad", [0, 1], ids=["vector", "scalar"])
def test_quant_special_blocks(zpp, block, pad):
    x = special_blocks(block)
    assert_quant_equal(run_quant_gpu(zpp, x, block, pad_src=pad),
                       oracle.quantize_blockwise_i8(x, block), "special block=%d" % block)


def test_quant_arbitrary_bit_patterns(zpp):
    x = synth.random_bits16(256 * 4096, 54)
    assert_quant_equal(run_quant_gpu(zpp, x, 256), oracle.quantize_blockwise_i8(x, 256), "bits")


def run_refresh_quant_gpu(zpp, x, block, pad_src=0, pad_dst=0, pad_codes=0):
    tx = to_dev(x, pad=pad_src)
    sec = empty_dev(x.size, np.uint16, pad=pad_dst, fill=0x7FC0)
    codes = empty_dev(x.size, np.int8, pad=pad_codes, fill=99)
    nb = (x.size + block - 1) // block
    scales = empty_dev(nb, np.float32, fill=-1.0)
    zpp.refresh_quantize_i8(sec, tx, codes, scales, block=block)
    torch.cuda.synchronize()
    return to_host(sec, np.uint16), to_host(codes, np.int8), to_host(scales, np.float32)


@pytest.mark.parametrize("block", [64, 192, 256, 320, 576, 960, 1024, 4032, 4096])
@pytest.mark.parametrize("n", [1, 7, 255, 256, 257, 256 * 5 + 80, 100000, 1 << 17])
def test_refresh_quantize_vs_oracle(zpp, block, n):
    """The refresh and its quantization in one pass: the secondary is the
    source bit for bit, codes and scales are the oracle's quantization."""
    x = synth.bf16_weights(n, 56, n + block)
    sec, codes, scales = run_refresh_quant_gpu(zpp, x, block)
    assert_bits_equal(sec, oracle.refresh(x), "secondary n=%d block=%d" % (n, block))
    assert_quant_equal((codes, scales), oracle.quantize_blockwise_i8(x, block),
                       "n=%d block=%d" % (n, block))


@pytest.mark.parametrize("pads", [(1, 0, 0), (0, 1, 0), (0, 0, 3), (8, 0, 0)],
                         ids=["src", "secondary", "codes", "src-16"])
def test_refresh_quantize_misaligned(zpp, pads):
    """Misaligned views take the scalar kernel (or, for a 16-byte-aligned
    offset, the vector one): the same bits."""
    n = 256 * 37 + 80
    x = synth.bf16_weights(n, 57)
    sec, codes, scales = run_refresh_quant_gpu(zpp, x, 256, *pads)
    assert_bits_equal(sec, x, "secondary pads=%s" % (pads,))
    assert_quant_equal((codes, scales), oracle.quantize_blockwise_i8(x, 256), "pads=%s" % (pads,))


@pytest.mark.parametrize("block", [256, 4032])
def test_refresh_quantize_special_blocks_and_bits(zpp, block):
    """Zero, Inf, NaN, tiny and huge blocks and arbitrary bit patterns (NaN
    payloads copied as they are)."""
    x = np.concatenate([special_blocks(block), synth.random_bits16(block * 64 + 33, 58)])
    sec, codes, scales = run_refresh_quant_gpu(zpp, x, block)
    assert_bits_equal(sec, x, "secondary")
    assert_quant_equal((codes, scales), oracle.quantize_blockwise_i8(x, block), "special")


# ===========================================================================
# Dequant-gather
# ===========================================================================
def run_gather_gpu(zpp, codes, scales, s, block, N, pad_out=0, code_pad=0):
    tc = [to_dev(c, pad=code_pad) for c in codes]
    ts = [to_dev(x) for x in scales]
    out = empty_dev(N, np.uint16, pad=pad_out, fill=0x5A5A)
    zpp.dequant_gather_layer(tc, ts, s, N, out, block=block)
    torch.cuda.synchronize()
    return to_host(out, np.uint16)


def quantized_shards(N, P2, block, cfg):
    s = secondary_elems(N, P2, block)
    w = np.zeros(P2 * s, np.uint16)
    w[:N] = synth.bf16_weights(N, cfg)
    qs = [oracle.quantize_blockwise_i8(w[j * s:(j + 1) * s], block) for j in range(P2)]
    return s, [q[0] for q in qs], [q[1] for q in qs]


def test_gather_tiny_layer(zpp):
    N, P2 = TINY.layer_elems, TINY.secondary_world
    s, codes, scales = quantized_shards(N, P2, 256, TINY.cfg_id)
    assert s == 2097152
    got = run_gather_gpu(zpp, codes, scales, s, 256, N)
    assert_bits_equal(got, oracle.dequant_gather_layer(codes, scales, s, 256, N), "tiny gather")


@pytest.mark.parametrize("P2,N,block", [
    (8, 8 * 8192 - 1152, 256),   # padded last shard, as in the Falcon-7B layer
    (8, 8 * 8192, 256),
    (1, 12345, 256),
    (3, 3 * 4096 - 4095, 64),    # last shard almost empty
    (64, 64 * 1024 - 1, 128),    # the largest secondary group
    (5, 5 * 2048 - 2048, 512),   # last shard entirely padding
    (2, 2 * 4096, 4096),
    (4, 4 * 6144 - 100, 2048),
    (3, 3 * 5120 - 1000, 1024),
    (8, 8 * 8192 - 1152, 192),   # blocks that are not powers of two
    (3, 3 * 5000 - 77, 320),
    (2, 2 * 4032 - 4031, 4032),
])
@pytest.mark.parametrize("pad_out", [0, 1], ids=["vector", "scalar"])
def test_gather_shapes(zpp, P2, N, block, pad_out):
    s, codes, scales = quantized_shards(N, P2, block, 60 + P2)
    got = run_gather_gpu(zpp, codes, scales, s, block, N, pad_out=pad_out)
    assert_bits_equal(got, oracle.dequant_gather_layer(codes, scales, s, block, N),
                      "P'=%d N=%d" % (P2, N))


@pytest.mark.parametrize("s", [1000, 256 * 3 + 8, 17])
def test_gather_unaligned_shard_length(zpp, s):
    """Shard lengths that are not a multiple of 16 take the scalar kernel;
    the last block of every shard is then short."""
    P2, block = 4, 256
    codes = [synth.random_codes(s, 61, j) for j in range(P2)]
    scales = [synth.random_scales((s + block - 1) // block, 61, j) for j in range(P2)]
    N = P2 * s - 5
    got = run_gather_gpu(zpp, codes, scales, s, block, N)
    assert_bits_equal(got, oracle.dequant_gather_layer(codes, scales, s, block, N), "s=%d" % s)


def test_gather_special_scales(zpp):
    P2, s, block = 2, 256 * 16, 256
    codes = [synth.random_codes(s, 62, j) for j in range(P2)]
    codes[0][:256] = 0
    scales = [synth.random_scales(s // block, 62, j) for j in range(P2)]
    scales[0][0] = np.inf        # 0 * inf = NaN and +-inf elsewhere
    scales[0][1] = np.nan
    scales[0][2] = 0.0
    scales[0][3] = -0.0
    scales[0][4] = 1e-40         # subnormal products
    scales[0][5] = 3e38          # overflow to +-inf
    scales[1][7] = np.float32(2.0 ** -133)
    for code_pad in (0, 3):
        got = run_gather_gpu(zpp, codes, scales, s, block, P2 * s, code_pad=code_pad)
        assert_bits_equal(got, oracle.dequant_gather_layer(codes, scales, s, block, P2 * s),
                          "special scales")


def test_gather_rounding_ties(zpp):
    """Every code against scales 2^e (1 + k 2^-9): many products fall exactly
    halfway between two bf16 values, so ties-to-even is exercised in the fast
    path (scales inside [2^-100, 2^100]) and in the generic one (outside)."""
    block = 256
    ks = np.arange(1, 129, dtype=np.float64)
    exps = [-133, -120, -101, -100, -30, 0, 7, 99, 100, 101, 110]
    sc = np.concatenate([(1.0 + ks * 2.0 ** -9) * 2.0 ** e for e in exps]).astype(np.float32)
    codes = np.tile(np.concatenate([np.arange(-128, 128, dtype=np.int16)]).astype(np.int8), sc.size)
    s = codes.size
    got = run_gather_gpu(zpp, [codes], [sc], s, block, s)
    assert_bits_equal(got, oracle.dequant_gather_layer([codes], [sc], s, block, s), "ties")


def test_gather_arbitrary_codes(zpp):
    P2, s, block = 8, 256 * 640, 256
    codes = [synth.random_codes(s, 63, j) for j in range(P2)]
    codes[2][::3] = -128  # outside the quantizer's range, still a valid input
    scales = [synth.random_scales(s // block, 63, j, lo=1e-30, hi=1e30) for j in range(P2)]
    N = P2 * s - 333
    got = run_gather_gpu(zpp, codes, scales, s, block, N)
    assert_bits_equal(got, oracle.dequant_gather_layer(codes, scales, s, block, N), "codes")


def test_gather_empty_layer_records_event(zpp):
    ev = zpp.Event()
    c = torch.zeros(256, dtype=torch.int8, device="cuda")
    sc = torch.zeros(1, dtype=torch.float32, device="cuda")
    out = torch.zeros(1, dtype=torch.int16, device="cuda")
    zpp.dequant_gather_layer([c], [sc], 256, 0, out, done_after=ev)
    ev.synchronize()
    assert ev.query()


# ===========================================================================
# Fused step + refresh + quantize
# ===========================================================================
def run_fused_gpu(zpp, p, m, v, g, hp, step, block, secondary=True, pad=0, pad_bf16=None,
                  pad_codes=None):
    tp, tm, tv, tg = (to_dev(x, pad=pad) for x in (p, m, v, g))
    n = p.size
    pb = pad if pad_bf16 is None else pad_bf16
    prim = empty_dev(n, np.uint16, pad=pb, fill=0x5555)
    sec = empty_dev(n, np.uint16, pad=pb, fill=0x7FC0) if secondary else None
    codes = empty_dev(n, np.int8, pad=pad if pad_codes is None else pad_codes, fill=99)
    scales = empty_dev((n + block - 1) // block, np.float32, fill=-1.0)
    zpp.adam_step_refresh_quantize(tp, tm, tv, tg, prim, sec, codes, scales, step=step,
                                   block=block, **hp)
    torch.cuda.synchronize()
    return (to_host(tp, np.float32), to_host(tm, np.float32), to_host(tv, np.float32),
            to_host(prim, np.uint16), to_host(sec, np.uint16) if secondary else None,
            to_host(codes, np.int8), to_host(scales, np.float32))


def assert_fused_matches_oracle(got, p, m, v, g, hp, step, block, what):
    gp, gm, gv, gb, gs, gc, gsc = got
    rp, rm, rv, rb = oracle.adam_step(p, m, v, g, step=step, **hp)
    assert_adam_close((gp, gm, gv, gb), (rp, rm, rv, rb), hp["lr"], what, prev=(p, m, v), g=g,
                      hp=hp)
    if gs is not None:
        assert_bits_equal(gs, gb, what + " secondary = primary")
    rc, rs = oracle.quantize_blockwise_i8(rb, block)
    n = p.size
    nb = (n + block - 1) // block
    same = np.array([np.array_equal(gb[k * block:(k + 1) * block], rb[k * block:(k + 1) * block])
                     for k in range(nb)])
    assert same.mean() > 0.95, what
    for k in np.nonzero(same)[0]:
        assert_bits_equal(gc[k * block:(k + 1) * block], rc[k * block:(k + 1) * block],
                          "%s codes block %d" % (what, k))
    assert_bits_equal(gsc[same], rs[same], what + " scales")


@pytest.mark.parametrize("block", [64, 128, 192, 256, 320, 512, 960, 1088, 2048, 2112, 4032,
                                   4096])
@pytest.mark.parametrize("n", [1, 255, 256, 4099, 1088 * 4 + 7, 256 * 40 + 80, 65536 + 64 + 3])
def test_fused_vs_oracle(zpp, block, n):
    hp = f32hp(HP_TINY)
    p = synth.master_weights(n, 70, n)
    g = synth.gradients(n, 70, n)
    m, v = synth.moments(n, 70, n)
    got = run_fused_gpu(zpp, p, m, v, g, hp, 2, block)
    assert_fused_matches_oracle(got, p, m, v, g, hp, 2, block, "n=%d block=%d" % (n, block))


@pytest.mark.parametrize("block", [192, 320, 1024, 4032])
def test_fused_two_kernel_blocks_misaligned_quantization(zpp, block):
    """Blocks other than 64-512 run the step with its copies, then the int8
    quantizer over the primary.  An 8-byte (not 16-byte) aligned primary and
    4-byte (not 8-byte) aligned codes keep the step's vector kernel but put
    the quantization on its scalar kernel: the same bits."""
    hp = f32hp(HP_TINY)
    n = block * 37 + 100
    p = synth.master_weights(n, 73, block)
    g = synth.gradients(n, 73, block)
    m, v = synth.moments(n, 73, block)
    got = run_fused_gpu(zpp, p, m, v, g, hp, 3, block, pad_bf16=4, pad_codes=4)
    assert_fused_matches_oracle(got, p, m, v, g, hp, 3, block, "block=%d" % block)


@pytest.mark.parametrize("secondary", [True, False], ids=["with-secondary", "no-secondary"])
@pytest.mark.parametrize("pad", [0, 1], ids=["fused", "scalar"])
@pytest.mark.parametrize("block", [256, 320])
def test_fused_equals_separate_calls(zpp, secondary, pad, block):
    """The fused entry gives, bit for bit, what the three separate calls give
    on the same inputs (both on the GPU), on both of its paths."""
    hp = f32hp(HP_LOUD)
    n = 256 * 300 + 17
    p = synth.master_weights(n, 71)
    g = synth.gradients(n, 71)
    m, v = synth.moments(n, 71)
    got = run_fused_gpu(zpp, p, m, v, g, hp, 5, block, secondary=secondary, pad=pad)
    tp, tm, tv, tg = (to_dev(x) for x in (p, m, v, g))
    prim = empty_dev(n, np.uint16)
    sec = empty_dev(n, np.uint16)
    codes = empty_dev(n, np.int8)
    scales = empty_dev((n + block - 1) // block, np.float32)
    zpp.adam_partition_step(tp, tm, tv, tg, prim, step=5, **hp)
    zpp.refresh_secondary(sec, prim)
    zpp.quantize_blockwise_i8(sec, codes, scales, block=block)
    torch.cuda.synchronize()
    sep = (to_host(tp, np.float32), to_host(tm, np.float32), to_host(tv, np.float32),
           to_host(prim, np.uint16), to_host(sec, np.uint16), to_host(codes, np.int8),
           to_host(scales, np.float32))
    for i, (a, b) in enumerate(zip(got, sep)):
        if a is not None:
            assert_bits_equal(a, b, "output %d" % i)
    assert_fused_matches_oracle(got, p, m, v, g, hp, 5, block, "fused")


def test_fused_special_values(zpp):
    """Non-finite gradients make a NaN weight; its block gets a NaN scale and
    zero codes, as the quantizer does for a NaN secondary."""
    hp = f32hp(HP_TINY)
    n, block = 256 * 8, 256
    p = synth.master_weights(n, 72)
    g = synth.gradients(n, 72)
    g[3 * 256 + 5] = np.nan
    g[6 * 256] = np.inf
    p[5 * 256:6 * 256] = 0.0
    g[5 * 256:6 * 256] = 0.0
    z = np.zeros(n, np.float32)
    got = run_fused_gpu(zpp, p, z, z, g, hp, 1, block)
    assert_fused_matches_oracle(got, p, z, z, g, hp, 1, block, "special")
    sc = got[6]
    assert np.isnan(sc[3]) and np.isnan(sc[6]) and sc[5] == 0.0
