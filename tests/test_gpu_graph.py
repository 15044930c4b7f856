"""The library under HIP graph capture: one iteration of the path (Adam step,
refresh, quantize on a second stream, gather on a third, ordered by the
library's events) is captured into a graph and replayed; every replay must
equal, bit for bit, the same iteration run eagerly from the same state.
The library allocates nothing and clears nothing with memsets, so nothing it
enqueues is illegal inside a capture."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2407_01614_amd import synth
from parity import assert_bits_equal, to_host

pytestmark = pytest.mark.gpu

HIP_CAPTURE_MODE_RELAXED = 2


@pytest.fixture(scope="module")
def zpp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2407_01614_amd import zpp as mod
    return mod


def hip():
    h = ctypes.CDLL("libamdhip64.so")
    P = ctypes.c_void_p
    h.hipStreamBeginCapture.argtypes = [P, ctypes.c_int]
    h.hipStreamEndCapture.argtypes = [P, ctypes.POINTER(P)]
    h.hipGraphInstantiate.argtypes = [ctypes.POINTER(P), P, P, P, ctypes.c_size_t]
    h.hipGraphLaunch.argtypes = [P, P]
    h.hipGraphExecDestroy.argtypes = [P]
    h.hipGraphDestroy.argtypes = [P]
    return h


@pytest.mark.parametrize("fused", [False, True, "copy"], ids=["separate", "fused", "fused-copy"])
def test_iteration_in_a_hip_graph(zpp, fused):
    n, B, P2 = (1 << 20) + 256, 256, 2
    hp = dict(lr=float(np.float32(1e-4)), beta1=float(np.float32(0.9)),
              beta2=float(np.float32(0.95)), eps=float(np.float32(1e-8)),
              weight_decay=float(np.float32(0.1)))
    p0 = torch.from_numpy(synth.master_weights(n, 110)).cuda()
    g = torch.from_numpy(synth.gradients(n, 110)).cuda()
    peer_c = synth.device_random_codes(n, 110, rank=1)
    peer_s = synth.device_random_scales(n // B, 110, rank=1)

    def state():
        return dict(p=p0.clone(), m=torch.zeros(n, device="cuda"), v=torch.zeros(n, device="cuda"),
                    prim=torch.empty(n, dtype=torch.int16, device="cuda"),
                    sec=torch.empty(n, dtype=torch.int16, device="cuda"),
                    codes=torch.empty(n, dtype=torch.int8, device="cuda"),
                    scales=torch.empty(n // B, dtype=torch.float32, device="cuda"),
                    out=torch.empty(P2 * n, dtype=torch.int16, device="cuda"))

    compute, copy, comm = torch.cuda.Stream(), torch.cuda.Stream(), torch.cuda.Stream()
    ev_prim, ev_quant, ev_gather = zpp.Event(), zpp.Event(), zpp.Event()

    def iteration(st):
        if fused == "copy":
            # the refresh and the quantization as one pass
            zpp.adam_partition_step(st["p"], st["m"], st["v"], g, st["prim"], step=1,
                                    stream=compute, **hp)
            ev_prim.record(compute)
            zpp.refresh_quantize_i8(st["sec"], st["prim"], st["codes"], st["scales"], block=B,
                                    stream=copy, wait_before=ev_prim, done_after=ev_quant)
        elif fused:
            ev_prim.record(compute)  # the fork: the second stream joins the capture here
            zpp.adam_step_refresh_quantize(st["p"], st["m"], st["v"], g, st["prim"], st["sec"],
                                           st["codes"], st["scales"], step=1, block=B,
                                           stream=copy, wait_before=ev_prim,
                                           done_after=ev_quant, **hp)
        else:
            zpp.adam_partition_step(st["p"], st["m"], st["v"], g, st["prim"], step=1,
                                    stream=compute, **hp)
            ev_prim.record(compute)
            zpp.refresh_secondary(st["sec"], st["prim"], stream=copy, wait_before=ev_prim)
            zpp.quantize_blockwise_i8(st["sec"], st["codes"], st["scales"], block=B,
                                      stream=copy, done_after=ev_quant)
        zpp.dequant_gather_layer([st["codes"], peer_c], [st["scales"], peer_s], n, P2 * n,
                                 st["out"], block=B, stream=comm, wait_events=[ev_quant],
                                 done_after=ev_gather)
        # join both side streams back into the one the capture started on
        zpp.stream_wait(compute, ev_quant)
        zpp.stream_wait(compute, ev_gather)

    def snapshot(st):
        return [to_host(st[k], np.uint8) for k in ("p", "m", "v", "prim", "sec", "codes",
                                                    "scales", "out")]

    # eager reference: the same iteration applied three times from the same state
    ref_state = state()
    torch.cuda.synchronize()
    refs = []
    for _ in range(3):
        iteration(ref_state)
        torch.cuda.synchronize()
        refs.append(snapshot(ref_state))

    h = hip()
    st = state()
    torch.cuda.synchronize()
    graph = ctypes.c_void_p()
    exe = ctypes.c_void_p()
    assert h.hipStreamBeginCapture(compute.cuda_stream, HIP_CAPTURE_MODE_RELAXED) == 0
    iteration(st)
    assert h.hipStreamEndCapture(compute.cuda_stream, ctypes.byref(graph)) == 0
    assert h.hipGraphInstantiate(ctypes.byref(exe), graph, None, None, 0) == 0
    try:
        for r in range(3):
            assert h.hipGraphLaunch(exe, compute.cuda_stream) == 0
            torch.cuda.synchronize()
            got = snapshot(st)
            for i, (a, b) in enumerate(zip(got, refs[r])):
                assert_bits_equal(a, b, "replay %d output %d" % (r, i))
            # eager work between replays
            torch.cuda.synchronize()
            _ = (st["p"].sum() + 1).item()
    finally:
        h.hipGraphExecDestroy(exe)
        h.hipGraphDestroy(graph)


@pytest.mark.parametrize("interleaved", [False, True], ids=["separate", "interleaved"])
@pytest.mark.parametrize("single_pass", [False, True], ids=["step", "single-pass"])
def test_receive_iteration_in_a_hip_graph(zpp, single_pass, interleaved):
    """An iteration that opens with the qgZ receive fused into the partition
    step (int4 gradient copies -> Adam), then the refresh, the quantization
    (or all three in the single receive pass) and the gather, on one stream,
    captured into a HIP graph and replayed three times with eager work in
    between: every replay equals the same iteration run eagerly from the same
    state, bit for bit.  `interleaved`: the int4 copies in one interleaved
    receive buffer, each written into its slots by the int4 quantizer."""
    n, B, P, P2 = (1 << 20) + 256, 256, 4, 2
    hp = dict(lr=float(np.float32(1e-4)), beta1=float(np.float32(0.9)),
              beta2=float(np.float32(0.95)), eps=float(np.float32(1e-8)),
              weight_decay=float(np.float32(0.1)))
    p0 = torch.from_numpy(synth.master_weights(n, 111)).cuda()
    src_c, src_s = [], []
    if interleaved:
        nc, ns = zpp.interleaved_sizes(n, B, P)
        il_c = torch.zeros(nc, dtype=torch.uint8, device="cuda")
        il_s = torch.zeros(ns, dtype=torch.float32, device="cuda")
    for q in range(P):
        g = synth.device_normal_f32(n, synth.GRAD_STD, 111, synth.KIND_GRAD, rank=q)
        if interleaved:
            zpp.quantize_blockwise_i4_interleaved(g, il_c, il_s, source=q, num_src=P, block=B)
            continue
        c = torch.empty((n + 1) // 2, dtype=torch.uint8, device="cuda")
        s = torch.empty((n + B - 1) // B, dtype=torch.float32, device="cuda")
        zpp.quantize_blockwise_i4(g, c, s, block=B)
        src_c.append(c)
        src_s.append(s)
    peer_c = synth.device_random_codes(n, 111, rank=1)
    peer_s = synth.device_random_scales(n // B, 111, rank=1)
    torch.cuda.synchronize()

    def state():
        return dict(p=p0.clone(), m=torch.zeros(n, device="cuda"), v=torch.zeros(n, device="cuda"),
                    prim=torch.empty(n, dtype=torch.int16, device="cuda"),
                    sec=torch.empty(n, dtype=torch.int16, device="cuda"),
                    codes=torch.empty(n, dtype=torch.int8, device="cuda"),
                    scales=torch.empty(n // B, dtype=torch.float32, device="cuda"),
                    out=torch.empty(P2 * n, dtype=torch.int16, device="cuda"))

    stream = torch.cuda.Stream()

    def iteration(st):
        if single_pass and interleaved:
            zpp.qgz_receive_step_refresh_quantize_interleaved(
                st["p"], st["m"], st["v"], il_c, il_s, P, st["prim"], st["sec"], st["codes"],
                st["scales"], step=1, grad_block=B, block=B, scale_out=1.0 / P, stream=stream,
                **hp)
        elif single_pass:
            zpp.qgz_receive_step_refresh_quantize(
                st["p"], st["m"], st["v"], src_c, src_s, st["prim"], st["sec"], st["codes"],
                st["scales"], step=1, grad_block=B, block=B, scale_out=1.0 / P, stream=stream,
                **hp)
        if not single_pass:
            if interleaved:
                zpp.qgz_receive_adam_step_interleaved(st["p"], st["m"], st["v"], il_c, il_s, P,
                                                      st["prim"], step=1, block=B,
                                                      scale_out=1.0 / P, stream=stream, **hp)
            else:
                zpp.qgz_receive_adam_step(st["p"], st["m"], st["v"], src_c, src_s, st["prim"],
                                          step=1, block=B, scale_out=1.0 / P, stream=stream,
                                          **hp)
            zpp.refresh_secondary(st["sec"], st["prim"], stream=stream)
            zpp.quantize_blockwise_i8(st["sec"], st["codes"], st["scales"], block=B,
                                      stream=stream)
        zpp.dequant_gather_layer([st["codes"], peer_c], [st["scales"], peer_s], n, P2 * n,
                                 st["out"], block=B, stream=stream)

    def snapshot(st):
        return [to_host(st[k], np.uint8) for k in ("p", "m", "v", "prim", "sec", "codes",
                                                    "scales", "out")]

    ref_state = state()
    torch.cuda.synchronize()
    refs = []
    for _ in range(3):
        iteration(ref_state)
        torch.cuda.synchronize()
        refs.append(snapshot(ref_state))

    h = hip()
    st = state()
    torch.cuda.synchronize()
    graph = ctypes.c_void_p()
    exe = ctypes.c_void_p()
    assert h.hipStreamBeginCapture(stream.cuda_stream, HIP_CAPTURE_MODE_RELAXED) == 0
    iteration(st)
    assert h.hipStreamEndCapture(stream.cuda_stream, ctypes.byref(graph)) == 0
    assert h.hipGraphInstantiate(ctypes.byref(exe), graph, None, None, 0) == 0
    try:
        for r in range(3):
            assert h.hipGraphLaunch(exe, stream.cuda_stream) == 0
            torch.cuda.synchronize()
            for i, (a, b) in enumerate(zip(snapshot(st), refs[r])):
                assert_bits_equal(a, b, "replay %d output %d" % (r, i))
            _ = (st["p"].sum() + 1).item()
    finally:
        h.hipGraphExecDestroy(exe)
        h.hipGraphDestroy(graph)
