"""The Python binding's own argument checks: the C ABI sees raw pointers
only, so the binding rejects what it cannot see (a tensor in host memory,
a wrong dtype, shape or stride, a pool smaller than the descriptor says)
with a Python exception, before anything is enqueued."""
import numpy as np
import pytest
import torch

from paper_2606_20474_amd import uq


def test_host_tensors_are_rejected():
    """Every entry point refuses tensors in host memory (no GPU needed)."""
    d = uq.CacheDesc(num_kv_heads=2, num_pages=4)
    r = uq.RefCacheDesc(num_kv_heads=2, num_pages=4, fmt="fp8")
    k = torch.zeros(3, 2, 128)
    q = torch.zeros(1, 4, 128)
    u8 = torch.zeros(1 << 16, dtype=torch.uint8)
    pt = torch.zeros(1, 4, dtype=torch.int32)
    ctx = torch.ones(1, dtype=torch.int32)
    pre = uq.SharedPrefix(torch.zeros(1, dtype=torch.int32), torch.zeros(1, dtype=torch.int32), 16)
    calls = [
        lambda: uq.quantize_kv(d, k, k, torch.zeros(3, dtype=torch.int64), u8, u8),
        lambda: uq.prepare_query(d, q),
        lambda: uq.quantize_error(k.reshape(-1, 128), torch.ones(1)),
        lambda: uq.decode_attention(d, q, u8, u8, pt, ctx, 16, workspace=u8),
        lambda: uq.decode_partials(d, q, u8, u8, pt, ctx, 16, 0.1, 0, u8, torch.zeros(1, 4, 128)),
        lambda: uq.decode_step(d, q, k[:1], k[:1], u8, u8, pt, ctx, 16, workspace=u8),
        lambda: uq.decode_merge(d, 1, 4, ctx, 16, 16, u8, torch.zeros(1, 4, 128)),
        lambda: uq.ref_write_kv(r, k, k, torch.zeros(3, dtype=torch.int64), u8),
        lambda: uq.ref_decode_attention(r, q, u8, pt, ctx, 16, workspace=u8),
        lambda: uq.ref_decode_step(r, q, k[:1], k[:1], u8, pt, ctx, 16, workspace=u8),
        lambda: uq.decode_cascade(d, q, u8, u8, pt, ctx, 16, pre, workspace=u8),
        lambda: uq.decode_cascade_merge(d, 1, 4, ctx, 16, pre, 16, u8, torch.zeros(1, 4, 128)),
        lambda: uq.ref_decode_cascade(r, q, u8, pt, ctx, 16, pre, workspace=u8),
    ]
    for i, call in enumerate(calls):
        with pytest.raises(ValueError, match="on the GPU"):
            call()


@pytest.fixture(scope="module")
def dev():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    return torch.device("cuda:0")


def setup(dev):
    d = uq.CacheDesc(num_kv_heads=2, num_pages=8)
    codes, scales = d.alloc_pools(dev, fill=0)
    g = torch.Generator(device=dev).manual_seed(3)
    k = torch.randn((20, 2, 128), generator=g, device=dev)
    slots = torch.arange(20, dtype=torch.int64, device=dev)
    q = torch.randn((2, 8, 128), generator=g, device=dev)
    pt = torch.tensor([[0, 1], [2, 3]], dtype=torch.int32, device=dev)
    ctx = torch.tensor([20, 5], dtype=torch.int32, device=dev)
    return d, codes, scales, k, slots, q, pt, ctx


@pytest.mark.gpu
def test_wrong_arguments_raise_before_any_launch(dev):
    d, codes, scales, k, slots, q, pt, ctx = setup(dev)
    bad = [
        (TypeError, lambda: uq.quantize_kv(d, k, k, slots.int(), codes, scales)),
        (ValueError, lambda: uq.quantize_kv(d, k[:, :1], k[:, :1], slots, codes, scales)),
        (ValueError, lambda: uq.quantize_kv(d, k, k[:, :, :64], slots, codes, scales)),
        (ValueError, lambda: uq.quantize_kv(d, k, k.transpose(1, 2).contiguous().transpose(1, 2), slots, codes,
                                            scales)),
        (ValueError, lambda: uq.quantize_kv(d, k, k, slots, codes[:100], scales)),
        (ValueError, lambda: uq.quantize_kv(d, k, k, slots[:5], codes, scales)),
        (TypeError, lambda: uq.decode_attention(d, q, codes, scales, pt.long(), ctx, 20)),
        (ValueError, lambda: uq.decode_attention(d, q, codes, scales, pt, ctx[:1], 20)),
        (ValueError, lambda: uq.decode_attention(d, q, codes, scales, pt[:1], ctx, 20)),
        (ValueError, lambda: uq.decode_attention(d, q.transpose(0, 1), codes, scales, pt, ctx, 20)),
        (ValueError, lambda: uq.decode_attention(d, q, codes, scales[:10], pt, ctx, 20)),
        (TypeError, lambda: uq.decode_attention(d, q, codes, scales, pt, ctx, 20,
                                                out=torch.empty((2, 8, 128), dtype=torch.float16, device=dev))),
        (ValueError, lambda: uq.decode_attention(d, q, codes, scales, pt, ctx, 20,
                                                 out=torch.empty((2, 8, 64), device=dev))),
        (ValueError, lambda: uq.decode_step(d, q, k[:2, :1], k[:2, :1], codes, scales, pt, ctx, 20)),
        (TypeError, lambda: uq.decode_step(d, q, k[:2], k[:2].half(), codes, scales, pt, ctx, 20)),
        (TypeError, lambda: uq.decode_cascade(d, q, codes, scales, pt, ctx, 20,
                                              uq.SharedPrefix(pt[0].clone(), ctx.long(), 16))),
        (ValueError, lambda: uq.decode_cascade(d, q, codes, scales, pt, ctx, 20,
                                               uq.SharedPrefix(pt[0, :0].clone(), ctx.clone(), 32))),
    ]
    for i, (exc, call) in enumerate(bad):
        print(f"bad call {i}", flush=True)
        with pytest.raises(exc):
            call()
    # the library is untouched: a valid write and decode still work
    uq.quantize_kv(d, k, k, slots, codes, scales)
    out = uq.decode_attention(d, q, codes, scales, pt, ctx, 20)
    torch.cuda.synchronize()
    assert torch.isfinite(out).all()
    assert (codes != 0).any()


@pytest.mark.gpu
def test_ref_cache_too_small(dev):
    r = uq.RefCacheDesc(num_kv_heads=2, num_pages=8, fmt="bf16")
    cache = r.alloc_cache(dev)
    k = torch.zeros((4, 2, 128), device=dev)
    with pytest.raises(ValueError):
        uq.ref_write_kv(r, k, k, torch.arange(4, device=dev), cache[:-1])


def test_write_page_table_row_length_is_bounded():
    """An explicit max_pages_per_seq longer than the page table's rows would
    make the write kernels read past the table: the binding refuses it
    before any other check (no GPU needed); 0 takes the row length."""
    pt = torch.zeros(2, 4, dtype=torch.int32)
    for bad in (5, 100, -1):
        with pytest.raises(ValueError, match="max_pages_per_seq"):
            uq._write_table(pt, bad)
    d = uq.CacheDesc(num_kv_heads=2, num_pages=4)
    r = uq.RefCacheDesc(num_kv_heads=2, num_pages=4, fmt="fp8")
    k = torch.zeros(3, 2, 128)
    slots = torch.zeros(3, dtype=torch.int64)
    u8 = torch.zeros(1 << 16, dtype=torch.uint8)
    with pytest.raises(ValueError, match="max_pages_per_seq"):
        uq.quantize_kv(d, k, k, slots, u8, u8, page_table=pt, max_pages_per_seq=5)
    with pytest.raises(ValueError, match="max_pages_per_seq"):
        uq.ref_write_kv(r, k, k, slots, u8, page_table=pt, max_pages_per_seq=5)
