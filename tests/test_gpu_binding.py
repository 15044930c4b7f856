"""The Python binding's argument handling on real device tensors: what the
binding itself rejects (type, device, dtype, layout, buffer sizes) and what
it passes on for the library to reject (block sizes, overlapping views of one
allocation, too many sources or events), each raising before anything is
enqueued; a size-0 call is a no-op."""
import pytest
import torch

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def zpp():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2407_01614_amd import zpp as mod
    return mod


HP = dict(lr=1e-4, beta1=0.9, beta2=0.95, eps=1e-8, weight_decay=0.1, step=1)


def f32(n):
    return torch.zeros(n, dtype=torch.float32, device="cuda")


def bf16(n):
    return torch.zeros(n, dtype=torch.int16, device="cuda")


def test_binding_rejects_bad_tensors(zpp):
    n = 1024
    p, m, v, g, o = f32(n), f32(n), f32(n), f32(n), bf16(n)
    with pytest.raises(TypeError):
        zpp.adam_partition_step(p.double(), m, v, g, o, **HP)
    with pytest.raises(TypeError):
        zpp.adam_partition_step(p.cpu().numpy(), m, v, g, o, **HP)
    with pytest.raises(ValueError):
        zpp.adam_partition_step(p.cpu(), m, v, g, o, **HP)
    with pytest.raises(ValueError):
        zpp.adam_partition_step(f32(2 * n)[::2], m, v, g, o, **HP)
    with pytest.raises(ValueError):
        zpp.adam_partition_step(p, m, v, g, bf16(n - 1), **HP)
    with pytest.raises(ValueError):
        zpp.refresh_secondary(bf16(n - 1), o)
    torch.cuda.synchronize()


def test_library_rejects_what_the_binding_passes_on(zpp):
    n = 1024
    src = bf16(n)
    codes = torch.zeros(n, dtype=torch.int8, device="cuda")
    scales = f32(n)  # room for any block count, so only the library's block check decides
    for block in (0, 100, 32, 8192):
        with pytest.raises(zpp.ZppError) as e:
            zpp.quantize_blockwise_i8(src, codes, scales, block=block)
        assert e.value.status == zpp.ZPP_EINVAL, block
    # two views of one allocation that share bytes
    buf = f32(3 * n)
    with pytest.raises(zpp.ZppError) as e:
        zpp.adam_partition_step(buf[:n], buf[n // 2:n // 2 + n], f32(n), f32(n), bf16(n), **HP)
    assert e.value.status == zpp.ZPP_EOVERLAP
    # a refresh onto its own source
    with pytest.raises(zpp.ZppError) as e:
        zpp.refresh_secondary(src, src)
    assert e.value.status == zpp.ZPP_EOVERLAP
    # hyperparameters
    with pytest.raises(zpp.ZppError) as e:
        zpp.adam_partition_step(f32(n), f32(n), f32(n), f32(n), bf16(n),
                                **dict(HP, step=0))
    assert e.value.status == zpp.ZPP_EINVAL
    torch.cuda.synchronize()


def test_source_and_event_limits(zpp):
    n, B = 512, 256
    c = torch.zeros((n + 1) // 2, dtype=torch.uint8, device="cuda")
    s = f32(n // B)
    out = f32(n)
    with pytest.raises(ValueError):
        zpp.dequant_reduce_i4([c] * (zpp.MAX_SHARDS + 1), [s] * (zpp.MAX_SHARDS + 1), n, out)
    with pytest.raises(ValueError):
        zpp.dequant_reduce_i4([], [], n, out)
    with pytest.raises(ValueError):
        zpp.dequant_reduce_i4([c, c], [s], n, out)
    events = [zpp.Event() for _ in range(zpp.MAX_WAIT_EVENTS + 1)]
    with pytest.raises(zpp.ZppError) as e:
        zpp.dequant_reduce_i4([c], [s], n, out, wait_events=events)
    assert e.value.status == zpp.ZPP_EINVAL
    torch.cuda.synchronize()


def test_size_zero_is_a_no_op(zpp):
    n = 256
    p = torch.full((n,), 1.5, device="cuda")
    o = torch.full((n,), 7, dtype=torch.int16, device="cuda")
    zpp.adam_partition_step(p, f32(n), f32(n), f32(n), o, n=0, **HP)
    zpp.refresh_secondary(o, bf16(n), count=0)
    torch.cuda.synchronize()
    assert bool((p == 1.5).all()) and bool((o == 7).all())
