"""Whole-array parity at the benchmarked shape: one step of the benchmark's
own pipeline (one stream, as timed; separate kernels, and the fused step +
refresh + quantize kernel in their place) at the Llama-2-13B rank partition
(203,372,880 elements) and layer (317,204,480 elements over 8 shards), with
every output copied back and compared in full with the oracle:

  * Adam master, moments and bf16 primary: the 1e-5 relative / 1 ulp bar,
    over all n elements;
  * the secondary: the primary, bit for bit;
  * the int8 codes and scales: the oracle's quantization of the GPU's own
    primary (identical inputs, so one correct result), bit for bit;
  * the gathered layer: the oracle's dequant-gather of the shards the GPU
    read, bit for bit.

The oracle runs on block-aligned ranges from a pool of host threads (its
calls release the GIL); the inputs are copied to the host before the step.
"""
import os
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle
from paper_2407_01614_amd.pipeline import PartitionPipeline
from paper_2407_01614_amd.workloads import WORKLOADS
from parity import ChunkedAdam, assert_bits_equal

pytestmark = pytest.mark.gpu

WL = WORKLOADS["llama-2-13b"]


@pytest.fixture(scope="module")
def zpp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2407_01614_amd import zpp as mod
    return mod


def threads():
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:
        return max(1, min(16, os.cpu_count() or 1))


def ranges(n, parts, align):
    step = max(align, -(-n // parts) // align * align)
    return [(a, min(n, a + step)) for a in range(0, n, step)]


def f32hp(hp):
    return {k: float(np.float32(v)) for k, v in hp.items()}


def h(t, dtype):
    return t.cpu().numpy().view(dtype)


@pytest.mark.parametrize("fused", [False, True], ids=["separate", "fused"])
def test_whole_arrays_one_step_llama2_13b(zpp, fused):
    n, B, s, N, P2 = WL.n, WL.block, WL.shard_elems, WL.layer_elems, WL.secondary_world
    hp = f32hp(WL.adam)
    pipe = PartitionPipeline(WL, streams=1, fused=fused)
    pipe.load_synthetic()
    p0, g = h(pipe.master, np.float32), h(pipe.grad, np.float32)
    peer_c = [h(c, np.int8) for c in pipe.peer_codes]
    peer_s = [h(x, np.float32) for x in pipe.peer_scales]
    pipe.step()
    pipe.wait()
    got_p, got_m, got_v = (h(t, np.float32) for t in (pipe.master, pipe.exp_avg, pipe.exp_avg_sq))
    got_b = h(pipe.primary, np.uint16)
    got_sec = h(pipe.secondary, np.uint16)
    got_c, got_s = h(pipe.codes, np.int8), h(pipe.scales, np.float32)
    got_out = h(pipe.out, np.uint16)
    del pipe
    torch.cuda.empty_cache()

    pool = ThreadPoolExecutor(threads())
    try:
        # Adam over the whole partition
        ref = ChunkedAdam(p0, hp, pool)
        ref.step(g)
        ref.check((got_p, got_m, got_v, got_b), "whole partition")
        del ref
        rs = ranges(n, 4 * threads(), B)
        # refresh
        assert_bits_equal(got_sec, got_b, "secondary = primary")
        # quantization of the GPU's own secondary, block by block
        q = list(pool.map(lambda r: oracle.quantize_blockwise_i8(got_sec[r[0]:r[1]], B), rs))
        assert_bits_equal(got_c, np.concatenate([x[0] for x in q]), "whole codes")
        assert_bits_equal(got_s, np.concatenate([x[1] for x in q]), "whole scales")
        del q
        # the gathered layer: local rank 0 = the first s codes of this rank's
        # quantized secondary, then the peers, each gathered into its place
        shard_c = [got_c[:s]] + peer_c
        shard_s = [got_s[:s // B]] + peer_s
        pieces = pool.map(lambda j: oracle.dequant_gather_layer(
            [shard_c[j]], [shard_s[j]], s, B, min(s, N - j * s)), range(P2))
        assert_bits_equal(got_out, np.concatenate(list(pieces)), "whole gathered layer")
    finally:
        pool.shutdown()
