"""Seeded synthetic inputs shaped like the paper's Llama-2 / Falcon workloads.

This module draws random numbers and nothing else: it holds none of the
partition path's arithmetic (no optimizer, no bf16 rounding rule, no
quantization).  Both the HIP path and the CPU oracle are fed from it.

Every array comes from ``numpy.random.default_rng(SeedSequence([cfg, kind,
rank, it]))`` so that a (config, kind, rank, iteration) tuple names one fixed
array on every machine.  ``kind`` is one of the constants below.
"""
import numpy as np

KIND_MASTER = 0
KIND_GRAD = 1
KIND_LAYER = 2
KIND_EXP_AVG = 3
KIND_EXP_AVG_SQ = 4
KIND_BITS = 5
KIND_CODES = 6
KIND_SCALES = 7

WEIGHT_STD = 0.02  # weights ~ N(0, 0.02)
GRAD_STD = 1e-3    # gradients ~ N(0, 1e-3)

_CHUNK = 1 << 24


def rng(cfg, kind, rank=0, it=0):
    return np.random.default_rng(np.random.SeedSequence([int(cfg), int(kind), int(rank), int(it)]))


def normal_f32(n, std, cfg, kind, rank=0, it=0):
    """n float32 draws from N(0, std^2), generated in chunks to bound memory."""
    g = rng(cfg, kind, rank, it)
    out = np.empty(n, np.float32)
    for lo in range(0, n, _CHUNK):
        hi = min(lo + _CHUNK, n)
        g.standard_normal(out=out[lo:hi], dtype=np.float32)
        out[lo:hi] *= np.float32(std)
    return out


def master_weights(n, cfg, rank=0):
    return normal_f32(n, WEIGHT_STD, cfg, KIND_MASTER, rank)


def gradients(n, cfg, rank=0, it=0):
    return normal_f32(n, GRAD_STD, cfg, KIND_GRAD, rank, it)


def moments(n, cfg, rank=0):
    """Non-zero Adam moments for tests that start past step 1: m ~ N(0, 1e-3)
    and v = (draw ~ N(0, 1e-3))^2, so that v >= 0."""
    m = normal_f32(n, GRAD_STD, cfg, KIND_EXP_AVG, rank)
    r = normal_f32(n, GRAD_STD, cfg, KIND_EXP_AVG_SQ, rank)
    return m, r * r


def bf16_weights(n, cfg, rank=0, it=0, std=WEIGHT_STD):
    """n bf16 bit patterns of weights ~ N(0, std^2): the high 16 bits of a
    float32 draw (truncation is just this generator's way of drawing bf16
    samples)."""
    f = normal_f32(n, std, cfg, KIND_LAYER, rank, it)
    return (f.view(np.uint32) >> np.uint32(16)).astype(np.uint16)


# --------------------------------------------------------------------------
# Device-side draws (torch's seeded GPU generator): same distributions, drawn
# in HBM directly, for the full-size workloads where host generation would
# dominate set-up time.  The host copies of what a test samples are taken
# from these tensors, so both sides still see identical inputs.
# --------------------------------------------------------------------------
def _device_gen(cfg, kind, rank, it, device):
    seed = int(np.random.SeedSequence([int(cfg), int(kind), int(rank), int(it)]).generate_state(1)[0])
    gen = torch_mod().Generator(device=device)
    gen.manual_seed(seed)
    return gen


def torch_mod():
    import torch
    return torch


def device_normal_f32(n, std, cfg, kind, rank=0, it=0, device="cuda"):
    torch = torch_mod()
    out = torch.empty(n, dtype=torch.float32, device=device)
    out.normal_(0.0, float(std), generator=_device_gen(cfg, kind, rank, it, device))
    return out


def device_bf16_weights(n, cfg, rank=0, it=0, std=WEIGHT_STD, device="cuda"):
    """bf16 bit patterns (as int16) of N(0, std^2) draws: the high halves of
    float32 draws, as in `bf16_weights`."""
    torch = torch_mod()
    f = device_normal_f32(n, std, cfg, KIND_LAYER, rank, it, device)
    return (f.view(torch.int32) >> 16).to(torch.int16)


def device_random_codes(n, cfg, rank=0, device="cuda"):
    """int8 codes uniform in [-127, 127], drawn on the device."""
    torch = torch_mod()
    return torch.randint(-127, 128, (n,), dtype=torch.int8, device=device,
                         generator=_device_gen(cfg, KIND_CODES, rank, 0, device))


def device_random_packed_i4(nbytes, cfg, rank=0, device="cuda"):
    """Arbitrary bytes, i.e. pairs of 4-bit two's-complement codes (every
    nibble from -8 to 7), drawn on the device."""
    torch = torch_mod()
    return torch.randint(0, 256, (nbytes,), dtype=torch.uint8, device=device,
                         generator=_device_gen(cfg, KIND_CODES, rank, 1, device))


def device_random_scales(nblocks, cfg, rank=0, lo=1e-5, hi=1e-3, device="cuda"):
    """Positive float32 scales, log-uniform in [lo, hi], drawn on the device."""
    torch = torch_mod()
    e = torch.empty(nblocks, dtype=torch.float64, device=device)
    e.uniform_(float(np.log(lo)), float(np.log(hi)),
               generator=_device_gen(cfg, KIND_SCALES, rank, 0, device))
    return e.exp().to(torch.float32)


def random_bits16(n, cfg, rank=0):
    """Arbitrary 16-bit patterns, NaN and Inf payloads included."""
    return rng(cfg, KIND_BITS, rank).integers(0, 1 << 16, size=n, dtype=np.uint16)


def random_codes(n, cfg, rank=0):
    """Arbitrary int8 codes in [-127, 127]."""
    return rng(cfg, KIND_CODES, rank).integers(-127, 128, size=n, dtype=np.int8)


def random_scales(nblocks, cfg, rank=0, lo=1e-5, hi=1e-3):
    """Positive float32 scales, log-uniform in [lo, hi]."""
    g = rng(cfg, KIND_SCALES, rank)
    e = g.uniform(np.log(lo), np.log(hi), size=nblocks)
    return np.exp(e).astype(np.float32)
