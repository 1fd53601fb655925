"""The Ultra-TQ comparison cache (format TQ4 of the comparison-cache calls)
on the GPU against the oracle's Ultra-TQ cache (appendix "Calibrated LUT
int4 KV Encoding (Ultra-TQ)"; readings T1-T5 in oracle/uq_oracle.c).

  * write: every byte of the cache (pre-filled with a canary) equal to the
    oracle's, for f32 and bf16 rows, padding slots, logical slots through a
    page table, the default and a calibrated (asymmetric) codebook;
  * decode: fp64 oracle attention over the oracle's cache, max-abs 2e-3 and
    relative L2 1e-3 (the query and the levels enter the matrix unit as the
    BF16 values both sides use, the values as their BF16 decode, so only the
    fp32 accumulation and the two-term P differ), ragged contexts, several
    partitions, group sizes 6, 16 and 1, and the Qwen3-235B-like layer at
    full size on sampled sequences;
  * the decode step and the cascade call run through the shared step and
    cascade tests with fmt "tq4".
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads
from paper_2606_20474_amd.codebook import default_tq_codebook

pytestmark = pytest.mark.gpu

SCALE = 1 / math.sqrt(128)
MAX_ABS = 2e-3
REL_L2 = 1e-3
CB = default_tq_codebook(128)
# a refit-style table: the theoretical levels compressed and shifted (asymmetric)
CB_CAL = (CB * np.float32(0.85) + np.float32(0.003)).astype(np.float32)


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


def physical_slots(wl, key, lo, hi, row):
    return wl.slots(key, lo, hi, row)


def fill_both(uq, wl, dev, codebook=CB, dtype=torch.float32):
    desc = uq.RefCacheDesc(wl.num_kv_heads, wl.num_pages, "tq4", codebook=codebook)
    cache = desc.alloc_cache(dev, fill=0x5A)
    ref = oracle.tq4_alloc_cache(wl.num_pages, wl.num_kv_heads, fill=0x5A)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev, dtype=dtype)
        slots = physical_slots(wl, key, lo, hi, row)
        uq.ref_write_kv(desc, k, v, torch.as_tensor(slots, device=dev), cache)
        oracle.tq4_write(k.float().cpu().numpy(), v.float().cpu().numpy(), slots, wl.num_pages, codebook, ref)
    return desc, cache, ref


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("which", ["default", "calibrated"])
def test_write_matches_oracle(uq, dtype, which):
    dev = torch.device("cuda:0")
    cb = CB if which == "default" else CB_CAL
    wl = workloads.custom(4, 8, 2, [5, 16, 33, 300], seed=51, paging="random")
    log(f"tq4 write {dtype} {which}")
    desc, cache, ref = fill_both(uq, wl, dev, cb, dtype)
    # padding slots and logical slots through a page table
    g = torch.Generator().manual_seed(5)
    k = torch.randn((6, wl.num_kv_heads, 128), generator=g).to(dtype)
    v = torch.randn((6, wl.num_kv_heads, 128), generator=g).to(dtype)
    logical = np.array([-1, 3, 16 * wl.max_pages_per_seq + 7, -1, 2 * 16 * wl.max_pages_per_seq + 40, 1], np.int64)
    uq.ref_write_kv(desc, k.to(dev), v.to(dev), torch.as_tensor(logical, device=dev), cache,
                    page_table=torch.as_tensor(wl.page_table, device=dev))
    phys = np.array([-1 if s < 0 else wl.page_table[s // (16 * wl.max_pages_per_seq),
                                                     (s % (16 * wl.max_pages_per_seq)) // 16] * 16 + s % 16
                     for s in logical], np.int64)
    oracle.tq4_write(k.float().numpy(), v.float().numpy(), phys, wl.num_pages, cb, ref)
    got = cache.cpu().numpy()
    diff = np.nonzero(got != ref)[0]
    assert diff.size == 0, f"{diff.size} bytes differ, first at {diff[:8]}"


@pytest.mark.parametrize("partition", [0, 32, 48, 64, 256])
def test_decode_against_oracle(uq, partition):
    dev = torch.device("cuda:0")
    wl = workloads.custom(6, 12, 2, [1, 17, 100, 257, 1000, 0], seed=52, paging="random")
    log(f"tq4 decode partition={partition}")
    desc, cache, ref = fill_both(uq, wl, dev)
    out = uq.ref_decode_attention(desc, wl.q.to(dev), cache, torch.as_tensor(wl.page_table, device=dev),
                                  torch.as_tensor(wl.context_lens, device=dev), wl.max_context, SCALE, partition)
    torch.cuda.synchronize()
    want = oracle.tq4_decode_attention(wl.q.numpy(), ref, wl.page_table, wl.context_lens, wl.num_kv_heads, CB)
    check(out.cpu().numpy(), want, f"tq4 p{partition}")
    assert np.all(out[5].cpu().numpy() == 0)


@pytest.mark.parametrize("hq,hkv", [(32, 2), (4, 4)])
def test_decode_group_sizes(uq, hq, hkv):
    dev = torch.device("cuda:0")
    wl = workloads.custom(3, hq, hkv, [40, 513, 96], seed=53, paging="random")
    log(f"tq4 decode hq={hq} hkv={hkv}")
    desc, cache, ref = fill_both(uq, wl, dev, CB_CAL)
    out = uq.ref_decode_attention(desc, wl.q.to(dev), cache, torch.as_tensor(wl.page_table, device=dev),
                                  torch.as_tensor(wl.context_lens, device=dev), wl.max_context, SCALE, 64)
    torch.cuda.synchronize()
    want = oracle.tq4_decode_attention(wl.q.numpy(), ref, wl.page_table, wl.context_lens, wl.num_kv_heads, CB_CAL)
    check(out.cpu().numpy(), want, f"tq4 {hq}/{hkv}")


def test_qwen_full_size_sampled(uq):
    """B=32, Hq=64, Hkv=4, context 32768, random pages, the default
    partition; two sequences against the oracle on a cache of their own."""
    dev = torch.device("cuda:0")
    wl = workloads.qwen3_235b_like()
    log("tq4 qwen3-235b-like full size")
    desc = uq.RefCacheDesc(wl.num_kv_heads, wl.num_pages, "tq4")
    cache = desc.alloc_cache(dev)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.ref_write_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), cache)
    out = uq.ref_decode_attention(desc, wl.q.to(dev), cache, torch.as_tensor(wl.page_table, device=dev),
                                  torch.as_tensor(wl.context_lens, device=dev), wl.max_context, SCALE, 0)
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    seqs = [0, 31]
    maxp = wl.max_pages_per_seq
    ptc = np.arange(len(seqs) * maxp, dtype=np.int32).reshape(len(seqs), maxp)
    ref = oracle.tq4_alloc_cache(len(seqs) * maxp, wl.num_kv_heads)
    for i, b in enumerate(seqs):
        for key, lo, hi in wl.sequence_segments(b):
            k, v = wl.kv(key, lo, hi, device=dev)
            pos = np.arange(lo, hi, dtype=np.int64)
            oracle.tq4_write(k.cpu().numpy(), v.cpu().numpy(), ptc[i, pos // 16].astype(np.int64) * 16 + pos % 16,
                             len(seqs) * maxp, CB, ref)
    want = oracle.tq4_decode_attention(wl.q.numpy()[seqs], ref, ptc, wl.context_lens[seqs], wl.num_kv_heads, CB)
    check(out[seqs], want, "tq4 qwen sampled")
