"""Cascade decode over a shared prefix (uq_decode_cascade and the comparison
caches' uq_ref_decode_cascade) through the C ABI.

The cascade calls compute the same attention as uq_decode_attention: the
shared prefix pages are read once per kv head for 16 (sequence, query head)
columns at a time, and the rest of each context through its page table,
then merged.  Checked against the fp64 oracle over the oracle's own cache
(max-abs 2e-3, relative L2 1e-3), against the non-cascade GPU result, and,
for the decode step, bit for bit against the separate write + cascade
decode.  Contexts shorter than the prefix (whose last page is a private
copy), equal to it, one token longer, much longer, and empty; prefix
partitions from one page pair up; group sizes 6, 16 and 1.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu

SCALE = 1 / math.sqrt(128)
MAX_ABS = 2e-3
REL_L2 = 1e-3


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def log(msg):
    print(msg, flush=True)


def check(got, ref, what, max_abs=MAX_ABS, rel_l2=REL_L2):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    log(f"{what}: max-abs {err.max():.3e} rel-L2 {rel:.3e}")
    assert np.all(np.isfinite(got)), what
    assert err.max() <= max_abs, (what, err.max())
    assert rel <= rel_l2, (what, rel)


def fill_fp4(uq, wl, dev, fill=0x5A):
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v)
    codes, scales = desc.alloc_pools(dev, fill=fill)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
    return desc, codes, scales


def prefix_of(uq, wl, dev, partition=0):
    return uq.SharedPrefix(torch.as_tensor(wl.prefix_pages.astype(np.int32), device=dev),
                           torch.as_tensor(wl.prefix_lens(), device=dev), wl.shared_prefix_tokens, partition)


def oracle_ref(wl, dev):
    pools = oracle.alloc_pools(wl.num_pages, wl.num_kv_heads)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), wl.slots(key, lo, hi, row), wl.num_pages,
                           rotate_v=wl.rotate_v, pools=pools)
    return oracle.decode_attention(wl.q.numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads, SCALE,
                                   wl.rotate_v)


def small(hq=12, hkv=2, seed=31):
    return workloads.custom(6, hq, hkv, [20, 96, 97, 150, 400, 0], seed=seed, paging="random",
                            shared_prefix_tokens=96)


@pytest.mark.parametrize("partition,prefix_partition", [(0, 0), (32, 32), (48, 32), (64, 64), (256, 32)])
def test_cascade_against_oracle(uq, partition, prefix_partition):
    dev = torch.device("cuda:0")
    wl = small()
    log(f"cascade G=6 partition={partition} prefix partition={prefix_partition}")
    desc, codes, scales = fill_fp4(uq, wl, dev)
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    pre = prefix_of(uq, wl, dev, prefix_partition)
    out = uq.decode_cascade(desc, q, codes, scales, pt, ctx, wl.max_context, pre, SCALE, partition)
    plain = uq.decode_attention(desc, q, codes, scales, pt, ctx, wl.max_context, SCALE, partition)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    check(out, oracle_ref(wl, dev), f"cascade p{partition}/{prefix_partition}")
    check(out, plain.cpu().numpy(), "cascade vs plain", 2e-4, 1e-5)
    assert np.all(out[5] == 0)


@pytest.mark.parametrize("hq,hkv", [(32, 2), (4, 4)])
def test_cascade_group_sizes(uq, hq, hkv):
    dev = torch.device("cuda:0")
    wl = small(hq, hkv, seed=32)
    log(f"cascade hq={hq} hkv={hkv}")
    desc, codes, scales = fill_fp4(uq, wl, dev)
    pre = prefix_of(uq, wl, dev, 32)
    out = uq.decode_cascade(desc, wl.q.to(dev), codes, scales, torch.as_tensor(wl.page_table, device=dev),
                            torch.as_tensor(wl.context_lens, device=dev), wl.max_context, pre, SCALE, 64)
    torch.cuda.synchronize()
    check(out.cpu().numpy(), oracle_ref(wl, dev), f"cascade {hq}/{hkv}")


@pytest.mark.parametrize("fmt", ["fp4", "fp8", "bf16", "tq4"])
def test_cascade_step_equals_write_then_cascade(uq, fmt):
    """The new token (after the prefix) written inside the cascade call."""
    dev = torch.device("cuda:0")
    wl = small(seed=33)
    log(f"cascade step {fmt}")
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    g = torch.Generator(device=dev).manual_seed(7)
    k_new = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g, device=dev)
    v_new = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g, device=dev)
    c = wl.context_lens.astype(np.int64)
    last = np.maximum(c - 1, 0)
    slots = wl.page_table[np.arange(wl.batch), last // 16].astype(np.int64) * 16 + last % 16
    slots = torch.as_tensor(np.where(c > 0, slots, -1), device=dev)
    pre = prefix_of(uq, wl, dev, 32)
    outs, pools = [], []
    for fused in (False, True):
        if fmt == "fp4":
            desc, codes, scales = fill_fp4(uq, wl, dev)
            if not fused:
                uq.quantize_kv(desc, k_new, v_new, slots, codes, scales)
            out = uq.decode_cascade(desc, q, codes, scales, pt, ctx, wl.max_context, pre, SCALE, 64,
                                    k_new=k_new if fused else None, v_new=v_new if fused else None)
            bufs = (codes, scales)
        else:
            desc = uq.RefCacheDesc(wl.num_kv_heads, wl.num_pages, fmt, 0.3, 0.3)
            cache = desc.alloc_cache(dev, fill=0x5A)
            for key, lo, hi, row in wl.segments():
                k, v = wl.kv(key, lo, hi, device=dev)
                uq.ref_write_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), cache)
            if not fused:
                uq.ref_write_kv(desc, k_new, v_new, slots, cache)
            out = uq.ref_decode_cascade(desc, q, cache, pt, ctx, wl.max_context, pre, SCALE, 64,
                                        k_new=k_new if fused else None, v_new=v_new if fused else None)
            bufs = (cache,)
        torch.cuda.synchronize()
        outs.append(out.cpu())
        pools.append([x.cpu().numpy() for x in bufs])
    for a, b in zip(*pools):
        assert np.array_equal(a, b), f"{fmt}: pools differ"
    assert torch.equal(outs[0], outs[1]), f"{fmt}: outputs differ"


def test_cascade_partials_plus_merge(uq):
    dev = torch.device("cuda:0")
    wl = small(seed=34)
    desc, codes, scales = fill_fp4(uq, wl, dev)
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    pre = prefix_of(uq, wl, dev)
    one = uq.decode_cascade(desc, q, codes, scales, pt, ctx, wl.max_context, pre, SCALE, 32)
    ws = torch.empty(uq.cascade_workspace_bytes(wl.num_kv_heads, wl.batch, wl.num_q_heads, wl.max_context, pre, 32),
                     dtype=torch.uint8, device=dev)
    two = torch.empty_like(q)
    uq.decode_cascade(desc, q, codes, scales, pt, ctx, wl.max_context, pre, SCALE, 32, workspace=ws, out=two,
                      partials_only=True)
    uq.decode_cascade_merge(desc, wl.batch, wl.num_q_heads, ctx, wl.max_context, pre, 32, ws, two)
    torch.cuda.synchronize()
    assert torch.equal(one, two)


def test_cascade_minimax_full_size_sampled(uq):
    """B=64, Hq=48, Hkv=8, lognormal contexts, 16k shared prefix, the
    default partitions: shortest and longest sequence against the oracle,
    and the whole batch against the non-cascade kernel."""
    dev = torch.device("cuda:0")
    wl = workloads.minimax_like()
    log("cascade minimax-like full size")
    desc, codes, scales = fill_fp4(uq, wl, dev, fill=None)
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    out = uq.decode_cascade(desc, q, codes, scales, pt, ctx, wl.max_context, prefix_of(uq, wl, dev), SCALE, 0)
    plain = uq.decode_attention(desc, q, codes, scales, pt, ctx, wl.max_context, SCALE, 0)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    check(out, plain.cpu().numpy(), "minimax cascade vs plain", 5e-4, 2e-5)
    seqs = [int(np.argmin(wl.context_lens)), int(np.argmax(wl.context_lens))]
    maxp = wl.max_pages_per_seq
    ptc = np.arange(len(seqs) * maxp, dtype=np.int32).reshape(len(seqs), maxp)
    pools = oracle.alloc_pools(len(seqs) * maxp, wl.num_kv_heads)
    for i, b in enumerate(seqs):
        for key, lo, hi in wl.sequence_segments(b):
            k, v = wl.kv(key, lo, hi, device=dev)
            pos = np.arange(lo, hi, dtype=np.int64)
            oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), ptc[i, pos // 16].astype(np.int64) * 16 + pos % 16,
                               len(seqs) * maxp, rotate_v=wl.rotate_v, pools=pools)
    ref = oracle.decode_attention(wl.q.numpy()[seqs], pools, ptc, wl.context_lens[seqs], wl.num_kv_heads, SCALE,
                                  wl.rotate_v)
    check(out[seqs], ref, "minimax cascade sampled")
