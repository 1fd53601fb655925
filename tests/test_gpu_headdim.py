"""The FP4 path at head sizes 64 and 256 (uq_cache_desc.head_dim) against
the oracle at the same head size.

  * quantize-on-write: every pool byte (pre-filled with a canary) equal to
    the oracle's, f32 and bf16 rows, rotate_v on and off, padding slots;
  * decode attention: max-abs 2e-3 and relative L2 1e-3 against the fp64
    oracle, ragged contexts with an empty one, partitions 0/32/48/256, group
    sizes 6, 16 and 1 (at head size 64 both the one-head and the two-head
    blocks), f32 and bf16 queries, a bf16 output, and a
    GPT-OSS-like layer (64 query heads, 8 KV heads, batch 32, context 32768)
    at full size on sampled sequences.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-3
REL_L2 = 1e-3


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def log(msg):
    print(msg, flush=True)


def check(got, ref, what):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    log(f"{what}: max-abs {err.max():.3e} rel-L2 {rel:.3e}")
    assert np.all(np.isfinite(got)), what
    assert err.max() <= MAX_ABS, (what, err.max())
    assert rel <= REL_L2, (what, rel)


def both_caches(uq, wl, dev, dtype=torch.float32, fill=0x5A):
    d = wl.head_dim
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v, head_dim=d)
    codes, scales = desc.alloc_pools(dev, fill=fill)
    pools = oracle.alloc_pools(wl.num_pages, wl.num_kv_heads, fill=fill if fill is not None else 0, head_dim=d)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev, dtype=dtype)
        slots = wl.slots(key, lo, hi, row)
        uq.quantize_kv(desc, k, v, torch.as_tensor(slots, device=dev), codes, scales)
        oracle.quantize_kv(k.float().cpu().numpy(), v.float().cpu().numpy(), slots, wl.num_pages,
                           rotate_v=wl.rotate_v, pools=pools)
    return desc, codes, scales, pools


def decode(uq, wl, desc, codes, scales, dev, partition=0, q=None, out_dtype=torch.float32):
    q = wl.q.to(dev) if q is None else q.to(dev)
    out = uq.decode_attention(desc, q, codes, scales, torch.as_tensor(wl.page_table, device=dev),
                              torch.as_tensor(wl.context_lens, device=dev), wl.max_context,
                              1 / math.sqrt(wl.head_dim), partition, out_dtype=out_dtype)
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


@pytest.mark.parametrize("d", [64, 256])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("rotate_v", [True, False])
def test_write_bit_exact(uq, d, dtype, rotate_v):
    dev = torch.device("cuda:0")
    wl = workloads.custom(4, 8, 2, [5, 16, 33, 300], seed=61, paging="random", rotate_v=rotate_v, head_dim=d)
    log(f"write d={d} {dtype} rotate_v={rotate_v}")
    desc, codes, scales, pools = both_caches(uq, wl, dev, dtype)
    g = torch.Generator().manual_seed(9)
    k = torch.randn((5, 2, d), generator=g).to(dtype)
    slots = np.array([-1, 3, 40, -7, 17], np.int64)
    uq.quantize_kv(desc, k.to(dev), (2 * k).to(dev), torch.as_tensor(slots, device=dev), codes, scales)
    oracle.quantize_kv(k.float().numpy(), (2 * k).float().numpy(), slots, wl.num_pages, rotate_v=rotate_v,
                       pools=pools)
    assert np.array_equal(codes.cpu().numpy(), pools[0]), "codes differ"
    assert np.array_equal(scales.cpu().numpy(), pools[1]), "scales differ"


@pytest.mark.parametrize("d", [64, 256])
@pytest.mark.parametrize("partition", [0, 32, 48, 256])
@pytest.mark.parametrize("rotate_v", [True, False])
def test_decode_ragged(uq, d, partition, rotate_v):
    dev = torch.device("cuda:0")
    wl = workloads.custom(6, 12, 2, [1, 17, 100, 257, 1000, 0], seed=62, paging="random", rotate_v=rotate_v,
                          head_dim=d)
    log(f"decode d={d} partition={partition} rotate_v={rotate_v}")
    desc, codes, scales, pools = both_caches(uq, wl, dev)
    out = decode(uq, wl, desc, codes, scales, dev, partition)
    ref = oracle.decode_attention(wl.q.numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads,
                                  1 / math.sqrt(d), rotate_v)
    assert np.all(out[5] == 0)
    check(out, ref, f"d={d} p={partition} rv={rotate_v}")


@pytest.mark.parametrize("d", [64, 256])
@pytest.mark.parametrize("hq,hkv", [(32, 2), (3, 3)])
def test_decode_group_sizes(uq, d, hq, hkv):
    dev = torch.device("cuda:0")
    wl = workloads.custom(3, hq, hkv, [40, 513, 96], seed=63, paging="random", head_dim=d)
    log(f"decode d={d} hq={hq} hkv={hkv}")
    desc, codes, scales, pools = both_caches(uq, wl, dev)
    out = decode(uq, wl, desc, codes, scales, dev, 64)
    ref = oracle.decode_attention(wl.q.numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads,
                                  1 / math.sqrt(d), True)
    check(out, ref, f"d={d} {hq}/{hkv}")


@pytest.mark.parametrize("hq,hkv,ctx", [(32, 4, [40, 513, 0, 2000]), (2, 2, [700, 1, 95, 4096]),
                                        (48, 8, [16, 17, 1000, 333])])
def test_decode_paired_heads(uq, hq, hkv, ctx):
    """Head size 64 with group size <= 8 and an even number of KV heads
    runs two KV heads per block (block-diagonal query operand): group sizes
    8, 1 and 6, an empty context, several partitions."""
    dev = torch.device("cuda:0")
    wl = workloads.custom(4, hq, hkv, ctx, seed=65, paging="random", head_dim=64)
    desc, codes, scales, pools = both_caches(uq, wl, dev)
    ref = oracle.decode_attention(wl.q.numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads,
                                  1 / math.sqrt(64), True)
    for partition in (0, 64, 512):
        log(f"paired d=64 hq={hq} hkv={hkv} partition={partition}")
        out = decode(uq, wl, desc, codes, scales, dev, partition)
        if 0 in ctx:
            assert np.all(out[ctx.index(0)] == 0)
        check(out, ref, f"paired {hq}/{hkv} p{partition}")


@pytest.mark.parametrize("d", [64, 256])
def test_decode_query_and_output_dtypes(uq, d):
    dev = torch.device("cuda:0")
    wl = workloads.custom(2, 8, 1, [700, 33], seed=64, paging="random", head_dim=d)
    desc, codes, scales, pools = both_caches(uq, wl, dev)
    qb = wl.q.bfloat16()
    ref_b = oracle.decode_attention(qb.float().numpy(), pools, wl.page_table, wl.context_lens, 1, 1 / math.sqrt(d),
                                    True)
    check(decode(uq, wl, desc, codes, scales, dev, q=qb), ref_b, f"d={d} bf16 q")
    ref = oracle.decode_attention(wl.q.numpy(), pools, wl.page_table, wl.context_lens, 1, 1 / math.sqrt(d), True)
    out_bf = decode(uq, wl, desc, codes, scales, dev, out_dtype=torch.bfloat16)
    # a bf16 output adds one rounding of the result (relative 2^-9)
    assert np.all(np.abs(out_bf - ref) <= MAX_ABS + np.abs(ref) * 2.0 ** -8)


@pytest.mark.parametrize("d", [64, 256])
def test_gpt_oss_like_full_size_sampled(uq, d):
    """64 query heads, 8 KV heads, batch 32, context 32768, random pages,
    the default partition; two sequences against the oracle."""
    dev = torch.device("cuda:0")
    wl = workloads.gpt_oss_like(d)
    log(f"decode {wl.name} full size")
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v, head_dim=d)
    codes, scales = desc.alloc_pools(dev)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
    out = decode(uq, wl, desc, codes, scales, dev)
    seqs = [3, 30]
    maxp = wl.max_pages_per_seq
    ptc = np.arange(len(seqs) * maxp, dtype=np.int32).reshape(len(seqs), maxp)
    pools = oracle.alloc_pools(len(seqs) * maxp, wl.num_kv_heads, head_dim=d)
    for i, b in enumerate(seqs):
        for key, lo, hi in wl.sequence_segments(b):
            k, v = wl.kv(key, lo, hi, device=dev)
            pos = np.arange(lo, hi, dtype=np.int64)
            oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), ptc[i, pos // 16].astype(np.int64) * 16 + pos % 16,
                               len(seqs) * maxp, rotate_v=wl.rotate_v, pools=pools)
    ref = oracle.decode_attention(wl.q.numpy()[seqs], pools, ptc, wl.context_lens[seqs], wl.num_kv_heads,
                                  1 / math.sqrt(d), wl.rotate_v)
    check(out[seqs], ref, f"{wl.name} sampled")
