"""The documented handling of device-resident indices that the host cannot
check (include/uq.h, "Conventions"): context lengths above max_context are
clamped to it, out-of-range page ids read page 0, and out-of-range or
negative write slots (and logical slots of sequences past num_seqs) write
nothing.  Each case is compared with the oracle on the equivalent in-range
inputs."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def caches(uq, wl, dev):
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v)
    codes, scales = desc.alloc_pools(dev, fill=0x3C)
    pools = oracle.alloc_pools(wl.num_pages, wl.num_kv_heads, fill=0x3C)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        slots = wl.slots(key, lo, hi, row)
        uq.quantize_kv(desc, k, v, torch.as_tensor(slots, device=dev), codes, scales)
        oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), slots, wl.num_pages, rotate_v=wl.rotate_v, pools=pools)
    return desc, codes, scales, pools


def decode(uq, desc, wl, codes, scales, dev, pt, ctx, max_context, partition):
    out = uq.decode_attention(desc, wl.q.to(dev), codes, scales, torch.as_tensor(pt, device=dev),
                              torch.as_tensor(ctx, device=dev), max_context, 1 / math.sqrt(128), partition)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def close(got, ref):
    err = np.abs(got - ref).max()
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    print(f"max-abs {err:.2e} rel-L2 {rel:.2e}", flush=True)
    assert err <= 2e-3 and rel <= 1e-3


@pytest.mark.parametrize("partition", [0, 64])
def test_context_above_max_context_is_clamped(uq, partition):
    dev = torch.device("cuda:0")
    wl = workloads.custom(3, 16, 2, [600, 300, 450], seed=81, paging="random")
    desc, codes, scales, pools = caches(uq, wl, dev)
    print(f"clamp: contexts above max_context, partition {partition}", flush=True)
    big = np.array([600, 5000, 100000], np.int32)      # above max_context = 450 for sequences 1 and 2
    got = decode(uq, desc, wl, codes, scales, dev, wl.page_table, big, 450, partition)
    ref = oracle.decode_attention(wl.q.numpy(), pools, wl.page_table, np.minimum(big, 450), wl.num_kv_heads,
                                  1 / math.sqrt(128), wl.rotate_v)
    close(got, ref)


def test_out_of_range_page_ids_read_page_zero(uq):
    dev = torch.device("cuda:0")
    wl = workloads.custom(2, 8, 1, [160, 96], seed=82, paging="random")
    desc, codes, scales, pools = caches(uq, wl, dev)
    print("clamp: page ids out of range", flush=True)
    pt = wl.page_table.copy()
    pt[0, 3] = wl.num_pages + 7          # inside sequence 0's context
    pt[1, 1] = -5                         # inside sequence 1's context
    pt_ref = pt.copy()
    pt_ref[0, 3] = 0
    pt_ref[1, 1] = 0
    got = decode(uq, desc, wl, codes, scales, dev, pt, wl.context_lens, wl.max_context, 32)
    ref = oracle.decode_attention(wl.q.numpy(), pools, pt_ref, wl.context_lens, wl.num_kv_heads, 1 / math.sqrt(128),
                                  wl.rotate_v)
    close(got, ref)


def test_write_slots_out_of_range_write_nothing(uq):
    dev = torch.device("cuda:0")
    desc = uq.CacheDesc(num_kv_heads=2, num_pages=4)
    codes, scales = desc.alloc_pools(dev, fill=0x77)
    print("clamp: write slots out of range", flush=True)
    g = torch.Generator().manual_seed(83)
    k = torch.randn((5, 2, 128), generator=g).to(dev)
    v = torch.randn((5, 2, 128), generator=g).to(dev)
    # physical slots: negative, one past the pool, far past it
    uq.quantize_kv(desc, k[:3], v[:3], torch.as_tensor([-1, 4 * 16, 10 ** 9], device=dev), codes, scales)
    torch.cuda.synchronize()
    assert torch.all(codes == 0x77) and torch.all(scales == 0x77)
    # logical slots through a page table: a sequence past num_seqs, a page id out of range
    pt = torch.as_tensor(np.array([[0, 1], [9, -2]], np.int32), device=dev)
    logical = torch.as_tensor([2 * 32 + 1, 32 + 0, 32 + 17], device=dev)   # seq 2 (none), seq 1 page 9, page -2
    uq.quantize_kv(desc, k[:3], v[:3], logical, codes, scales, page_table=pt)
    torch.cuda.synchronize()
    assert torch.all(codes == 0x77) and torch.all(scales == 0x77)
