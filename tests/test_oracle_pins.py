"""Pins of the CPU oracle against things other than itself.

Each check takes an ``Oracle`` instance so that ``test_oracle_mutants.py`` can
run the same checks against builds of the oracle with a planted mistake and
see them fail.  Pins used:
  * bf16 rounding: torch's CPU float32 -> bfloat16 conversion (a library RNE
    routine), exhaustive over all 2^16 bf16 patterns for the reverse way;
  * Adam: the closed form of step 1 from zero moments (m_hat = g,
    v_hat = g^2), the same closed form at any step from any moments when
    both betas are 0, and torch.optim.AdamW / Adam (float64, single-tensor
    path) as an independent implementation at arbitrary steps and states;
  * quantization: exact integer constructions (codes known in advance),
    power-of-two scaling, ties-to-even cases, sign symmetry, an error bound
    checked in exact rational arithmetic, special blocks;
  * dequant/gather: library float32 products and library bf16 rounding,
    marker shards, concatenation and round-trip bounds;
  * partition sizes: hand-worked values in ``tests/golden``.
"""
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

import oracle
from paper_2407_01614_amd import synth

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")

F32_MAX_BITS = 0x7F7FFFFF


def ulp_diff_f32(a, b):
    """Distance in units of last place between float32 arrays (ordered ints)."""
    ai = np.asarray(a, np.float32).view(np.int32).astype(np.int64)
    bi = np.asarray(b, np.float32).view(np.int32).astype(np.int64)
    ai = np.where(ai < 0, -(ai & 0x7FFFFFFF), ai)
    bi = np.where(bi < 0, -(bi & 0x7FFFFFFF), bi)
    return np.abs(ai - bi)


def torch_bf16_bits(x_f32):
    t = torch.from_numpy(np.ascontiguousarray(x_f32, np.float32)).to(torch.bfloat16)
    return t.view(torch.int16).numpy().view(np.uint16)


def bf16_of(values):
    """Exact bf16 bit patterns of values that bf16 represents exactly."""
    f = np.asarray(values, np.float32)
    bits = (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)
    back = (bits.astype(np.uint32) << np.uint32(16)).view(np.float32)
    assert np.array_equal(back, f), "value not exact in bf16"
    return bits


def trunc_bits(values):
    """bf16 bit patterns made by keeping the high half of float32 values."""
    f = np.ascontiguousarray(values, np.float32)
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# ===========================================================================
# bf16 conversions
# ===========================================================================
def special_f32():
    bits = [0x00000000, 0x80000000, 0x00000001, 0x007FFFFF, 0x00800000, 0x00008000,
            0x00018000, 0x00017FFF, 0x00018001, 0x3F800000, 0x3F808000, 0x3F818000,
            0x3F807FFF, 0x3F808001, 0xBF808000, 0xBF818000, 0x7F7F7FFF, 0x7F7F8000,
            0x7F7FFFFF, 0xFF7F8000, 0xFF7FFFFF, 0x7F800000, 0xFF800000, 0x477FE000,
            0x477FF000, 0x0000FFFF, 0x8000FFFF, 0x00FF8000, 0x00FE8000]
    return np.array(bits, np.uint32).view(np.float32)


def check_bf16_rne(orc):
    rng = np.random.default_rng(1234)
    rand_bits = rng.integers(0, 1 << 32, size=1 << 21, dtype=np.uint64).astype(np.uint32)
    # force a share of exact ties and near-ties
    ties = (rng.integers(0, 1 << 16, size=1 << 16, dtype=np.uint32) << np.uint32(16)) | np.uint32(0x8000)
    near = ties + rng.integers(-2, 3, size=ties.size).astype(np.uint32)
    x = np.concatenate([special_f32(), rand_bits.view(np.float32), ties.view(np.float32),
                        near.view(np.float32),
                        rng.standard_normal(1 << 18).astype(np.float32) * np.float32(0.02)])
    finite_or_inf = ~np.isnan(x)
    got = orc.bf16_rne(x)
    ref = torch_bf16_bits(x)
    assert np.array_equal(got[finite_or_inf], ref[finite_or_inf])
    # NaN: canonical quiet NaN with the sign dropped, whatever the payload
    assert np.all(got[~finite_or_inf] == 0x7FC0)
    assert (~finite_or_inf).sum() > 1000


def test_bf16_rne_matches_library():
    check_bf16_rne(oracle.default())


def test_bf16_rne_nan_payloads_canonical():
    nans = np.array([0x7FC00000, 0xFFC00000, 0x7F800001, 0xFF800001, 0x7FFFFFFF, 0x7FBFFFFF],
                    np.uint32).view(np.float32)
    assert np.all(oracle.bf16_rne(nans) == 0x7FC0)


def test_bf16_ties_to_even_by_hand():
    # 1 + 2^-8 is halfway between 1 and 1 + 2^-7: even neighbour is 1.0
    # 1 + 3*2^-8 is halfway between 1 + 2^-7 and 1 + 2^-6: even is 1 + 2^-6
    # (2 - 2^-8) * 2^127 is halfway between the largest bf16 (odd) and 2^128:
    # it rounds to infinity
    x = np.array([1 + 2.0 ** -8, 1 + 3 * 2.0 ** -8, -(1 + 2.0 ** -8), (2 - 2.0 ** -8) * 2.0 ** 127],
                 np.float32)
    assert list(oracle.bf16_rne(x)) == [0x3F80, 0x3F82, 0xBF80, 0x7F80]


def check_bf16_to_f32(orc):
    allbits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    got = orc.bf16_to_f32(allbits).view(np.uint32)
    ref = torch.from_numpy(allbits.view(np.int16)).view(torch.bfloat16).float().numpy().view(np.uint32)
    assert np.array_equal(got, ref)


def test_bf16_to_f32_exhaustive():
    check_bf16_to_f32(oracle.default())


# ===========================================================================
# Adam(W) partition step
# ===========================================================================
# hyperparameters of the Tiny workload (lr 1e-4, betas 0.9/0.95, eps 1e-8, wd 0.1)
HP_TINY = dict(lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1)
# exaggerated settings under which weight decay and eps placement are visible
HP_LOUD = dict(lr=1e-2, beta1=0.8, beta2=0.9, eps=1e-6, weight_decay=0.5)


def f32(x):
    return float(np.float32(x))


def hp32(hp):
    return {k: f32(v) for k, v in hp.items()}


def step1_closed_form(p0, g, hp):
    """From m = v = 0 at t = 1: m_hat = g and v_hat = g^2 exactly, so
    p1 = p0 (1 - lr wd) - lr g / (|g| + eps), m1 = (1 - b1) g, v1 = (1 - b2) g^2."""
    lr, b1, b2, eps, wd = (hp[k] for k in ("lr", "beta1", "beta2", "eps", "weight_decay"))
    p0 = p0.astype(np.float64)
    g = g.astype(np.float64)
    p1 = p0 * (1.0 - lr * wd) - lr * g / (np.abs(g) + eps)
    return p1, (1.0 - b1) * g, (1.0 - b2) * g * g


def check_adam_step1_closed_form(orc):
    rng = np.random.default_rng(7)
    n = 1 << 14
    for hp in (hp32(HP_TINY), hp32(HP_LOUD)):
        p0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
        # gradients spanning 1e-9 .. 1e-2, some exactly zero, some at |g| ~ eps
        g = (rng.standard_normal(n) * 10.0 ** rng.uniform(-9, -2, n)).astype(np.float32)
        g[::97] = 0.0
        g[1::89] = np.float32(hp["eps"]) * rng.choice([-1, 1], size=g[1::89].size)
        z = np.zeros(n, np.float32)
        p1, m1, v1, out = orc.adam_step(p0, z, z, g, step=1, **hp)
        ep, em, ev = step1_closed_form(p0, g, hp)
        assert ulp_diff_f32(p1, ep.astype(np.float32)).max() <= 1
        assert ulp_diff_f32(m1, em.astype(np.float32)).max() <= 1
        assert ulp_diff_f32(v1, ev.astype(np.float32)).max() <= 1
        assert np.array_equal(out, torch_bf16_bits(p1))


def test_adam_step1_closed_form():
    check_adam_step1_closed_form(oracle.default())


def check_adam_zero_betas_closed_form(orc):
    """With beta1 = beta2 = 0 the moments are the step's own gradient and its
    square and both bias corrections are 1, so any step t from any moments
    reduces to the step-1 closed form (with m1 = g', v1 = g'^2, where g' is
    the gradient, plus wd p0 in the L2 form)."""
    rng = np.random.default_rng(17)
    n = 1 << 12
    base = hp32(HP_LOUD)
    hp = dict(base, beta1=0.0, beta2=0.0)
    for adamw in (True, False):
        for t in (1, 2, 7, 1000):
            p0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
            g = (rng.standard_normal(n) * 10.0 ** rng.uniform(-6, -2, n)).astype(np.float32)
            m0 = (rng.standard_normal(n) * 1e-3).astype(np.float32)
            v0 = (rng.standard_normal(n) * 1e-3).astype(np.float32) ** 2
            p1, m1, v1, _ = orc.adam_step(p0, m0, v0, g, step=t, adamw=adamw, **hp)
            lr, eps, wd = hp["lr"], hp["eps"], hp["weight_decay"]
            p64, g64 = p0.astype(np.float64), g.astype(np.float64)
            if adamw:
                gg = g64
                ep = p64 * (1.0 - lr * wd) - lr * gg / (np.abs(gg) + eps)
            else:
                gg = g64 + wd * p64
                ep = p64 - lr * gg / (np.abs(gg) + eps)
            assert ulp_diff_f32(p1, ep.astype(np.float32)).max() <= 1, (adamw, t)
            assert ulp_diff_f32(m1, gg.astype(np.float32)).max() <= 1, (adamw, t)
            assert ulp_diff_f32(v1, (gg * gg).astype(np.float32)).max() <= 1, (adamw, t)


def test_adam_zero_betas_closed_form():
    check_adam_zero_betas_closed_form(oracle.default())


def test_adam_zero_grad_only_decays():
    hp = hp32(HP_LOUD)
    p0 = (np.random.default_rng(3).standard_normal(4096) * 0.02).astype(np.float32)
    z = np.zeros_like(p0)
    p1, m1, v1, _ = oracle.adam_step(p0, z, z, z, step=1, **hp)
    exact = [Fraction(float(p)) * (1 - Fraction(hp["lr"]) * Fraction(hp["weight_decay"]))
             for p in p0[:256]]
    assert ulp_diff_f32(p1[:256], np.array([float(e) for e in exact], np.float32)).max() <= 1
    assert not m1.any() and not v1.any()


def torch_adam_reference(p, m, v, g, hp, step, adamw):
    """One step of torch.optim.AdamW (or Adam with L2 decay) in float64 from
    the given state; step is the 1-based t the step is taken at."""
    pt = torch.nn.Parameter(torch.from_numpy(p.astype(np.float64)))
    cls = torch.optim.AdamW if adamw else torch.optim.Adam
    opt = cls([pt], lr=hp["lr"], betas=(hp["beta1"], hp["beta2"]), eps=hp["eps"],
              weight_decay=hp["weight_decay"], foreach=False, fused=False)
    pt.grad = torch.from_numpy(g.astype(np.float64))
    opt.state[pt] = {"step": torch.tensor(float(step - 1), dtype=torch.float64),
                     "exp_avg": torch.from_numpy(m.astype(np.float64)),
                     "exp_avg_sq": torch.from_numpy(v.astype(np.float64))}
    opt.step()
    st = opt.state[pt]
    return (pt.detach().numpy().astype(np.float32), st["exp_avg"].numpy().astype(np.float32),
            st["exp_avg_sq"].numpy().astype(np.float32))


def check_adam_vs_torch(orc):
    n = 4096
    for adamw in (True, False):
        for hp in (hp32(HP_TINY), hp32(HP_LOUD)):
            for t in (1, 2, 7, 100, 5000):
                p = synth.master_weights(n, cfg=90 + t, rank=int(adamw))
                g = synth.gradients(n, cfg=90 + t, rank=int(adamw))
                m, v = synth.moments(n, cfg=90 + t, rank=int(adamw))
                if t == 1:
                    m[:] = 0
                    v[:] = 0
                rp, rm, rv = torch_adam_reference(p, m, v, g, hp, t, adamw)
                op, om, ov, _ = orc.adam_step(p, m, v, g, step=t, adamw=adamw, **hp)
                assert ulp_diff_f32(op, rp).max() <= 1, (adamw, hp, t)
                assert ulp_diff_f32(om, rm).max() <= 1, (adamw, hp, t)
                assert ulp_diff_f32(ov, rv).max() <= 1, (adamw, hp, t)


def test_adam_vs_torch_optim():
    check_adam_vs_torch(oracle.default())


def check_adam_multistep_vs_torch(orc):
    """20 steps; torch keeps float64 state, so its state is brought back to the
    stored float32 values after every step, as the partition keeps it."""
    n = 64
    hp = hp32(HP_LOUD)
    p = synth.master_weights(n, cfg=5)
    m = np.zeros(n, np.float32)
    v = np.zeros(n, np.float32)
    tp, tm, tv = p.copy(), m.copy(), v.copy()
    for t in range(1, 21):
        g = synth.gradients(n, cfg=5, it=t) * np.float32(10.0)
        p, m, v, out = orc.adam_step(p, m, v, g, step=t, **hp)
        tp, tm, tv = torch_adam_reference(tp, tm, tv, g, hp, t, True)
        assert ulp_diff_f32(p, tp).max() <= 2, t
        assert ulp_diff_f32(m, tm).max() <= 2, t
        assert ulp_diff_f32(v, tv).max() <= 2, t
        assert np.array_equal(out, torch_bf16_bits(p))
        tp, tm, tv = p.copy(), m.copy(), v.copy()


def test_adam_multistep_vs_torch():
    check_adam_multistep_vs_torch(oracle.default())


def test_adam_emits_bf16_of_stored_master():
    hp = hp32(HP_TINY)
    n = 1 << 16
    p = synth.master_weights(n, cfg=11)
    g = synth.gradients(n, cfg=11)
    z = np.zeros(n, np.float32)
    p1, _, _, out = oracle.adam_step(p, z, z, g, step=1, **hp)
    assert np.array_equal(out, torch_bf16_bits(p1))
    _, _, _, none = oracle.adam_step(p, z, z, g, step=1, emit=False, **hp)
    assert none is None


def test_adam_nonfinite_grad_propagates():
    hp = hp32(HP_TINY)
    p = np.full(4, 0.01, np.float32)
    g = np.array([np.inf, -np.inf, np.nan, 0.0], np.float32)
    z = np.zeros(4, np.float32)
    p1, m1, v1, out = oracle.adam_step(p, z, z, g, step=1, **hp)
    assert np.isnan(p1[:3]).all() and np.isfinite(p1[3])
    assert np.all(out[:3] == 0x7FC0)


# ===========================================================================
# Secondary refresh
# ===========================================================================
def check_refresh(orc):
    for n in (0, 1, 7, 4099):
        src = synth.random_bits16(n, cfg=21, rank=n)
        dst = orc.refresh(src)
        assert dst.dtype == np.uint16 and np.array_equal(dst, src)


def test_refresh_is_bit_copy():
    check_refresh(oracle.default())


# ===========================================================================
# Blockwise int8 quantization
# ===========================================================================
def int_block(rng, block, with_extreme=True):
    q = rng.integers(-127, 128, size=block).astype(np.int8)
    if with_extreme:
        q[rng.integers(0, block)] = rng.choice([-127, 127])
    return q


def check_quant_integer_blocks(orc):
    """Blocks whose values are k * 2^e with |k| <= 127 and max |k| = 127: the
    scale must be 2^e exactly and the codes must be the k, at every exponent
    bf16 can hold the block exactly (subnormal blocks included)."""
    rng = np.random.default_rng(5)
    for block in (64, 192, 256, 320, 4096):
        exps = list(range(-133, 121, 7)) + [-126, -107, -100, -99, 0, 120]
        q = np.concatenate([int_block(rng, block) for _ in exps])
        x = np.concatenate([q[i * block:(i + 1) * block].astype(np.float64) * 2.0 ** e
                            for i, e in enumerate(exps)]).astype(np.float32)
        codes, scales = orc.quantize_blockwise_i8(bf16_of(x), block)
        assert np.array_equal(codes, q), block
        assert np.array_equal(scales, np.array([2.0 ** e for e in exps], np.float32)), block


def test_quant_integer_blocks():
    check_quant_integer_blocks(oracle.default())


def check_quant_ties_to_even(orc):
    # absmax 127 gives scale 1 and inverse 1, so the code is rint(x) itself
    vals = [127.0, 0.5, 1.5, 2.5, 3.5, -0.5, -1.5, -2.5, 126.5, -126.5, 0.25, 0.75, -0.75]
    expect = [127, 0, 2, 2, 4, 0, -2, -2, 126, -126, 0, 1, -1]
    x = np.zeros(64, np.float32)
    x[:len(vals)] = vals
    codes, scales = orc.quantize_blockwise_i8(bf16_of(x), 64)
    assert scales[0] == 1.0
    assert list(codes[:len(vals)]) == expect


def test_quant_ties_to_even():
    check_quant_ties_to_even(oracle.default())


def exact(f):
    return Fraction(float(f))


def check_quant_nearest_code(orc):
    """For random N(0, 0.02) blocks: max |x| maps to +-127, the scale is the
    float32 nearest absmax/127 (checked against the exact quotient), and every
    code is the nearest integer to x/scale up to the rounding slack of the
    scale and the inverse (at most 381 * 2^-24 of a scale, bounded here by
    2^-15).  Checked in exact rational arithmetic."""
    rng = np.random.default_rng(11)
    block = 64
    x = (rng.standard_normal(block * 40) * 0.02).astype(np.float32)
    xb = trunc_bits(x)
    codes, scales = orc.quantize_blockwise_i8(xb, block)
    xf = (xb.astype(np.uint32) << np.uint32(16)).view(np.float32)
    slack = Fraction(1, 1 << 15)
    for k in range(40):
        blk = xf[k * block:(k + 1) * block]
        a = np.abs(blk).max()
        sc = exact(scales[k])
        q_exact = exact(a) / 127
        # correctly rounded: no float32 neighbour is closer
        up = exact(np.nextafter(scales[k], np.float32(np.inf)))
        dn = exact(np.nextafter(scales[k], np.float32(0)))
        assert abs(sc - q_exact) <= abs(up - q_exact) and abs(sc - q_exact) <= abs(dn - q_exact)
        cb = codes[k * block:(k + 1) * block].astype(int)
        assert np.abs(cb[np.abs(blk) == a]).min() == 127
        for xi, ci in zip(blk, cb):
            err = abs(exact(xi) - ci * sc)
            assert err <= sc * (Fraction(1, 2) + slack)
            for other in (ci - 1, ci + 1):
                if -127 <= other <= 127:
                    assert abs(exact(xi) - other * sc) >= sc * (Fraction(1, 2) - slack)


def test_quant_nearest_code_exact():
    check_quant_nearest_code(oracle.default())


def check_quant_symmetry_and_scaling(orc):
    x = synth.bf16_weights(256 * 33 + 80, cfg=31)
    codes, scales = orc.quantize_blockwise_i8(x, 256)
    ncodes, nscales = orc.quantize_blockwise_i8(x ^ np.uint16(0x8000), 256)
    assert np.array_equal(ncodes, -codes) and np.array_equal(nscales, scales)
    xf = (x.astype(np.uint32) << np.uint32(16)).view(np.float32)
    for e in (-90, -40, -7, 3, 30, 60):
        xs = bf16_of((xf.astype(np.float64) * 2.0 ** e).astype(np.float32))
        c2, s2 = orc.quantize_blockwise_i8(xs, 256)
        assert np.array_equal(c2, codes), e
        assert np.array_equal(s2, (scales.astype(np.float64) * 2.0 ** e).astype(np.float32)), e


def test_quant_sign_symmetry_and_pow2_scaling():
    check_quant_symmetry_and_scaling(oracle.default())


def check_quant_special_blocks(orc):
    block = 64
    x = np.zeros(block * 6 + 10, np.float32)
    rng = np.random.default_rng(2)
    x[block:] = rng.standard_normal(x.size - block) * 0.02
    x[2 * block + 5] = np.inf
    x[3 * block + 9] = -np.inf
    x[4 * block + 63] = np.nan
    xb = trunc_bits(x)
    xb[4 * block + 63] = 0x7FC1  # a NaN with a payload
    codes, scales = orc.quantize_blockwise_i8(xb, block)
    assert scales.size == 7
    assert scales[0] == 0.0 and not codes[:block].any()
    sbits = scales.view(np.uint32)
    for k in (2, 3, 4):
        assert sbits[k] == 0x7FC00000, k
        assert not codes[k * block:(k + 1) * block].any()
    for k in (1, 5):
        assert np.isfinite(scales[k]) and scales[k] > 0
    # the short tail block takes its absmax from its own 10 elements only
    tail = (xb[6 * block:].astype(np.uint32) << np.uint32(16)).view(np.float32)
    assert scales[6] == np.float32(np.abs(tail).max()) / np.float32(127)
    assert np.abs(codes[6 * block:]).max() == 127


def test_quant_special_blocks():
    check_quant_special_blocks(oracle.default())


def check_quant_block_boundaries(orc):
    """Block k scaled by 2^k: each block's scale is its own, so an off-by-one
    in the block index shows up as a wrong scale or code."""
    rng = np.random.default_rng(9)
    for block in (64, 128, 192, 256, 320, 512, 4032):
        nb = 9
        q = np.concatenate([int_block(rng, block) for _ in range(nb)])
        q = q[:nb * block - 17]  # short last block (still contains its own extreme?)
        q[-1] = 127
        x = np.concatenate([q[k * block:(k + 1) * block].astype(np.float64) * 2.0 ** (k - 4)
                            for k in range(nb)]).astype(np.float32)
        codes, scales = orc.quantize_blockwise_i8(bf16_of(x), block)
        assert np.array_equal(codes, q), block
        assert np.array_equal(scales, np.array([2.0 ** (k - 4) for k in range(nb)], np.float32))


def test_quant_block_boundaries():
    check_quant_block_boundaries(oracle.default())


def test_quant_empty():
    codes, scales = oracle.quantize_blockwise_i8(np.zeros(0, np.uint16), 256)
    assert codes.size == 0 and scales.size == 0


# ===========================================================================
# Dequantization and the gather
# ===========================================================================
def check_dequant_vs_library(orc):
    n = 256 * 40 + 100
    codes = synth.random_codes(n, cfg=41)
    scales = synth.random_scales(oracle.num_blocks(n, 256), cfg=41)
    scales[3] = np.float32(np.nan)
    scales[4] = 0.0
    scales[5] = np.float32(3e38)  # products overflow to inf in float32
    scales[6] = np.float32(1e-40)  # subnormal scale
    got = orc.dequant_blockwise_i8(codes, scales, 256)
    with np.errstate(over="ignore", invalid="ignore"):
        prod = codes.astype(np.float32) * np.repeat(scales, 256)[:n]
    ref = torch_bf16_bits(prod)
    isn = np.isnan(prod)
    assert np.array_equal(got[~isn], ref[~isn])
    assert np.all(got[isn] == 0x7FC0) and isn.sum() == 256


def test_dequant_vs_library():
    check_dequant_vs_library(oracle.default())


def check_gather_markers(orc):
    """Shard j holds code (j+1) everywhere with scale 2^-j: the gathered layer
    must read (j+1)*2^-j on exactly [j*s, (j+1)*s), cut at N."""
    for P2, s, N in ((8, 1024, 8 * 1024 - 300), (2, 512, 1024), (3, 256, 600), (1, 768, 700)):
        codes = [np.full(s, j + 1, np.int8) for j in range(P2)]
        scales = [np.full(s // 256, 2.0 ** -j, np.float32) for j in range(P2)]
        out = orc.dequant_gather_layer(codes, scales, s, 256, N)
        assert out.size == N
        expect = np.concatenate([np.full(s, (j + 1) * 2.0 ** -j, np.float32)
                                 for j in range(P2)])[:N]
        assert np.array_equal(out, bf16_of(expect))


def test_gather_markers():
    check_gather_markers(oracle.default())


def check_gather_is_concatenation(orc):
    P2, block = 4, 256
    N = 4 * 2048 - 1000
    s = oracle.secondary_shard_elems(N, P2, block)
    codes = [synth.random_codes(s, cfg=51, rank=j) for j in range(P2)]
    scales = [synth.random_scales(s // block, cfg=51, rank=j) for j in range(P2)]
    out = orc.dequant_gather_layer(codes, scales, s, block, N)
    cat = np.concatenate([orc.dequant_blockwise_i8(c, sc, block)
                          for c, sc in zip(codes, scales)])[:N]
    assert np.array_equal(out, cat)
    # P' = 1 is the plain dequantization
    one = orc.dequant_gather_layer(codes[:1], scales[:1], s, block, s)
    assert np.array_equal(one, orc.dequant_blockwise_i8(codes[0], scales[0], block))


def test_gather_is_concatenation():
    check_gather_is_concatenation(oracle.default())


def check_round_trip(orc):
    """quantize -> gather returns each weight within half a scale (plus the
    slack) before the final bf16 rounding, i.e. within that plus half a bf16
    ulp of the result."""
    N, P2, block = 3 * 4096 + 1000, 4, 256
    w = synth.bf16_weights(N, cfg=61)
    s = oracle.secondary_shard_elems(N, P2, block)
    padded = np.zeros(P2 * s, np.uint16)
    padded[:N] = w
    qs = [orc.quantize_blockwise_i8(padded[j * s:(j + 1) * s], block) for j in range(P2)]
    out = orc.dequant_gather_layer([q[0] for q in qs], [q[1] for q in qs], s, block, N)
    wf = (w.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    with np.errstate(invalid="ignore"):  # a planted mistake may return non-integers
        of = (out.astype(np.uint32) << np.uint32(16)).view(np.float32).astype(np.float64)
    sc = np.concatenate([np.repeat(q[1], block)[:s] for q in qs])[:N].astype(np.float64)
    bound = sc * (0.5 + 2.0 ** -15) + np.abs(of) * 2.0 ** -8
    assert np.all(np.abs(wf - of) <= bound)


def test_round_trip_bound():
    check_round_trip(oracle.default())


# ===========================================================================
# Partition sizes (Eq. 1)
# ===========================================================================
def golden_shapes():
    rows = []
    with open(os.path.join(GOLDEN, "workload_shapes.txt")) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                kind, name, *nums = line.split()
                rows.append((kind, name, *map(int, nums)))
    return rows


@pytest.mark.parametrize("row", golden_shapes(), ids=lambda r: r[0] + "-" + r[1])
def test_partition_sizes_golden(row):
    kind, name, total, world, block, size, extra, blocks = row
    if kind == "layer":
        assert oracle.secondary_shard_elems(total, world, block) == size
        assert world * size - total == extra
        assert oracle.num_blocks(size, block) == blocks
        b, e = oracle.secondary_slice(total, world, world - 1, block)
        assert e == total and e - b == size - extra
    else:
        b, e = oracle.primary_slice(total, world, 1)
        assert (b, e - b) == (size, size)
        assert size % block == extra
        assert oracle.num_blocks(size, block) == blocks


# ===========================================================================
# qgZ: int4 gradient quantization and the dequantize-and-reduce
# ===========================================================================
def check_i4_packing(orc):
    """Hand-worked bytes: codes (1, -1) -> 0xF1, (7, -7) -> 0x97, (0, 2) ->
    0x20, (2, -2) -> 0xE2 (element 2i in the low nibble, two's complement);
    an odd tail leaves the high nibble 0."""
    x = np.array([1, -1, 7, -7, 0.5, 1.5, 2.5, -2.5, 3.0], np.float32)
    codes, scales = orc.quantize_blockwise_i4(x, 64)
    assert scales.tolist() == [1.0]
    assert codes.tolist() == [0xF1, 0x97, 0x20, 0xE2, 0x03]
    assert orc.unpack_i4(codes, 9).tolist() == [1, -1, 7, -7, 0, 2, 2, -2, 3]


def test_i4_packing_by_hand():
    check_i4_packing(oracle.default())


def i4_block(rng, block):
    q = rng.integers(-7, 8, size=block).astype(np.int8)
    q[rng.integers(0, block)] = rng.choice([-7, 7])
    return q


def check_i4_integer_blocks(orc):
    rng = np.random.default_rng(15)
    for block in (64, 256, 1024):
        exps = list(range(-149, 121, 9)) + [-126, -101, -100, 0, 120]
        q = np.concatenate([i4_block(rng, block) for _ in exps])
        x = np.concatenate([q[i * block:(i + 1) * block].astype(np.float64) * 2.0 ** e
                            for i, e in enumerate(exps)]).astype(np.float32)
        codes, scales = orc.quantize_blockwise_i4(x, block)
        assert np.array_equal(orc.unpack_i4(codes, x.size), q), block
        assert np.array_equal(scales, np.array([2.0 ** e for e in exps], np.float32)), block


def test_i4_integer_blocks():
    check_i4_integer_blocks(oracle.default())


def check_i4_ties_and_specials(orc):
    vals = [7.0, 0.5, 1.5, 2.5, 3.5, -0.5, -1.5, 6.5, -6.5]
    x = np.zeros(64 * 5 + 3, np.float32)
    x[:len(vals)] = vals
    x[64:128] = 0.0                       # zero block
    x[128:192] = np.linspace(-1, 1, 64)
    x[130] = np.inf                       # non-finite block
    x[192:256] = np.linspace(-3, 3, 64)
    x[200] = np.nan
    x[256:320] = np.linspace(-0.5, 0.25, 64)
    x[320:] = [1e-3, -4e-3, 2e-3]         # short tail block
    codes, scales = orc.quantize_blockwise_i4(x, 64)
    c = orc.unpack_i4(codes, x.size)
    assert c[:len(vals)].tolist() == [7, 0, 2, 2, 4, 0, -2, 6, -6]
    assert scales[1] == 0.0 and not c[64:128].any()
    assert scales.view(np.uint32)[2] == 0x7FC00000 and not c[128:192].any()
    assert scales.view(np.uint32)[3] == 0x7FC00000 and not c[192:256].any()
    assert scales[5] == np.float32(4e-3) / np.float32(7) and c[320:].tolist() == [2, -7, 4]
    n2 = orc.quantize_blockwise_i4(-x, 64)
    assert np.array_equal(orc.unpack_i4(n2[0], x.size), -c)


def test_i4_ties_and_specials():
    check_i4_ties_and_specials(oracle.default())


def check_i4_nearest_code(orc):
    rng = np.random.default_rng(16)
    block = 64
    x = (rng.standard_normal(block * 30) * 1e-3).astype(np.float32)
    codes, scales = orc.quantize_blockwise_i4(x, block)
    c = orc.unpack_i4(codes, x.size).astype(int)
    slack = Fraction(1, 1 << 15)
    for k in range(30):
        blk = x[k * block:(k + 1) * block]
        a = np.abs(blk).max()
        sc = exact(scales[k])
        qx = exact(a) / 7
        up = exact(np.nextafter(scales[k], np.float32(np.inf)))
        dn = exact(np.nextafter(scales[k], np.float32(0)))
        assert abs(sc - qx) <= abs(up - qx) and abs(sc - qx) <= abs(dn - qx)
        cb = c[k * block:(k + 1) * block]
        assert np.abs(cb[np.abs(blk) == a]).min() == 7
        for xi, ci in zip(blk, cb):
            assert abs(exact(xi) - ci * sc) <= sc * (Fraction(1, 2) + slack)
            for other in (ci - 1, ci + 1):
                if -7 <= other <= 7:
                    assert abs(exact(xi) - other * sc) >= sc * (Fraction(1, 2) - slack)


def test_i4_nearest_code_exact():
    check_i4_nearest_code(oracle.default())


def f32_round_exact(r):
    """The binary32 value nearest the rational r (ties to even), by exact
    comparison with the neighbours of a candidate."""
    cand = np.float32(float(r))
    best = None
    for c in (np.nextafter(cand, np.float32(-np.inf)), cand, np.nextafter(cand, np.float32(np.inf))):
        d = abs(exact(c) - r)
        if best is None or d < best[0] or (d == best[0] and (c.view(np.uint32) & 1) == 0):
            best = (d, c)
    return best[1]


def check_i4_dequant_reduce(orc):
    rng = np.random.default_rng(17)
    n, block, P = 64 * 12 + 5, 64, 4
    srcs = [(rng.standard_normal(n) * 10.0 ** rng.uniform(-5, -2, n)).astype(np.float32)
            for _ in range(P)]
    q = [orc.quantize_blockwise_i4(s, block) for s in srcs]
    codes = [orc.unpack_i4(c, n).astype(int) for c, _ in q]
    # brute force in exact rationals: acc = RN(code * s + acc) per source, then RN(acc * f)
    f = np.float32(0.25)
    out = orc.dequant_reduce_i4([c for c, _ in q], [s for _, s in q], n, block, float(f))
    for i in range(0, n, 7):
        acc = np.float32(0.0)
        for j in range(P):
            acc = f32_round_exact(codes[j][i] * exact(q[j][1][i // block]) + exact(acc))
        want = f32_round_exact(exact(acc) * exact(f))
        assert out[i].view(np.uint32) == want.view(np.uint32), i
    # one source, unit output scale: the dequantized partition (a float32 product)
    one = orc.dequant_reduce_i4([q[0][0]], [q[0][1]], n, block, 1.0)
    prod = codes[0].astype(np.float32) * np.repeat(q[0][1], block)[:n]
    assert np.array_equal(one.view(np.uint32), prod.view(np.uint32))
    # integer sums are exact whatever the order: P copies of an integer block
    ints = np.concatenate([i4_block(rng, block) for _ in range(4)]).astype(np.float32)
    ci, si = orc.quantize_blockwise_i4(ints, block)
    tot = orc.dequant_reduce_i4([ci] * 8, [si] * 8, ints.size, block, 0.125)
    assert np.array_equal(tot, ints)


def test_i4_dequant_reduce_brute_force():
    check_i4_dequant_reduce(oracle.default())


@pytest.mark.parametrize("part", range(16))
def test_bf16_rne_exhaustive_vs_library(part):
    """Every float32 bit pattern (a sixteenth per case): the oracle's rounding
    equals torch's CPU conversion on all non-NaN values, and every NaN gives
    the canonical 0x7FC0."""
    orc = oracle.default()
    span = 1 << 28
    for lo in range(part * span, (part + 1) * span, 1 << 25):
        bits = np.arange(lo, lo + (1 << 25), dtype=np.uint32)
        x = bits.view(np.float32)
        got = orc.bf16_rne(x)
        ref = torch_bf16_bits(x)
        isnan = (bits & np.uint32(0x7FFFFFFF)) > np.uint32(0x7F800000)
        assert np.array_equal(got[~isnan], ref[~isnan]), hex(lo)
        assert np.all(got[isnan] == 0x7FC0), hex(lo)
