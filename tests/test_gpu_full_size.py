"""Every sequence of the full-size workloads against the oracle, in the launch
configuration the benchmark times.

* qwen3-235b-like (B = 32, Hq = 64, Hkv = 4, every context 32768, random
  pages, the default partition): decode attention, and the fused decode step
  (each sequence's new K/V token written at its last position, then
  attention over the context ending with it), for all 32 sequences.
* minimax-like (B = 64, Hq = 48, Hkv = 8, lognormal contexts 8k..128k, a
  16k-token prefix shared by every sequence, read once per kv head by the
  cascade call): the cascade decode step for all 64 sequences.

The oracle quantises the same seeded K/V (and new tokens) itself, a few
sequences at a time, and computes fp64 attention; the bar is max-abs 2e-3
and relative L2 1e-3 (Algorithm 1, Decode)."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-3
REL_L2 = 1e-3
CHUNK = 8   # sequences per oracle pass (bounds host memory)


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def log(msg):
    print(msg, flush=True)


def new_tokens(wl, seed):
    """The step's new K and V token of every sequence, fp32 [B, Hkv, 128] on the CPU."""
    g = torch.Generator().manual_seed(seed)
    k = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g)
    v = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g)
    return k, v


def oracle_outputs(wl, dev, new=None):
    """fp64 oracle attention of every sequence (with `new` = (k, v): after the
    step's token is written at position len - 1), CHUNK sequences at a time."""
    out = np.zeros((wl.batch, wl.num_q_heads, 128))
    maxp = wl.max_pages_per_seq
    for c0 in range(0, wl.batch, CHUNK):
        seqs = list(range(c0, min(c0 + CHUNK, wl.batch)))
        pt = np.arange(len(seqs) * maxp, dtype=np.int32).reshape(len(seqs), maxp)
        pools = oracle.alloc_pools(len(seqs) * maxp, wl.num_kv_heads)
        for i, b in enumerate(seqs):
            for key, lo, hi in wl.sequence_segments(b):
                k, v = wl.kv(key, lo, hi, device=dev)
                pos = np.arange(lo, hi, dtype=np.int64)
                slots = pt[i, pos // 16].astype(np.int64) * 16 + pos % 16
                oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), slots, len(seqs) * maxp, rotate_v=wl.rotate_v,
                                   pools=pools)
                del k, v
            if new is not None and wl.context_lens[b] > 0:
                last = int(wl.context_lens[b]) - 1
                slot = np.array([int(pt[i, last // 16]) * 16 + last % 16], dtype=np.int64)
                oracle.quantize_kv(new[0][b:b + 1].numpy(), new[1][b:b + 1].numpy(), slot, len(seqs) * maxp,
                                   rotate_v=wl.rotate_v, pools=pools)
        out[seqs] = oracle.decode_attention(wl.q.numpy()[seqs], pools, pt, wl.context_lens[seqs], wl.num_kv_heads,
                                            1 / math.sqrt(128), wl.rotate_v)
        log(f"  oracle: sequences {seqs[0]}..{seqs[-1]} done")
    return out


def gpu_cache(uq, wl, dev):
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v)
    codes, scales = desc.alloc_pools(dev)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
        del k, v
    torch.cuda.synchronize()
    return desc, codes, scales


def check(got, ref, what):
    got = np.asarray(got, np.float64)
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    worst = np.unravel_index(np.argmax(err), err.shape)
    log(f"{what}: max-abs {err.max():.3e} at (b, h, c) = {worst}, rel-L2 {rel:.3e}")
    assert np.all(np.isfinite(got)), what
    assert err.max() <= MAX_ABS, (what, err.max(), worst)
    assert rel <= REL_L2, (what, rel)
    # every sequence within the bar on its own, too
    for b in range(got.shape[0]):
        rb = np.linalg.norm(got[b] - ref[b]) / np.linalg.norm(ref[b])
        assert rb <= REL_L2, (what, b, rb)


def test_qwen_decode_every_sequence(uq):
    dev = torch.device("cuda:0")
    wl = workloads.qwen3_235b_like()
    log("qwen3-235b-like full size: decode, every sequence against the oracle")
    desc, codes, scales = gpu_cache(uq, wl, dev)
    out = uq.decode_attention(desc, wl.q.to(dev), codes, scales, torch.as_tensor(wl.page_table, device=dev),
                              torch.as_tensor(wl.context_lens, device=dev), wl.max_context, 1 / math.sqrt(128))
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    del codes, scales
    torch.cuda.empty_cache()
    check(out, oracle_outputs(wl, dev), "qwen decode, 32 sequences")


def test_qwen_step_every_sequence(uq):
    """The fused step the benchmark times (uq_decode_step, default partition):
    each sequence's new token at position 32767, then attention over the
    context that ends with it."""
    dev = torch.device("cuda:0")
    wl = workloads.qwen3_235b_like()
    log("qwen3-235b-like full size: decode step, every sequence against the oracle")
    desc, codes, scales = gpu_cache(uq, wl, dev)
    kn, vn = new_tokens(wl, 12345)
    out = uq.decode_step(desc, wl.q.to(dev), kn.to(dev), vn.to(dev), codes, scales,
                         torch.as_tensor(wl.page_table, device=dev), torch.as_tensor(wl.context_lens, device=dev),
                         wl.max_context, 1 / math.sqrt(128))
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    del codes, scales
    torch.cuda.empty_cache()
    check(out, oracle_outputs(wl, dev, new=(kn, vn)), "qwen decode step, 32 sequences")


def test_minimax_cascade_step_every_sequence(uq):
    """The cascade decode step the benchmark times on the minimax-like layer
    (shared prefix read once per kv head, default partitions, new tokens
    written into each sequence's private last page)."""
    dev = torch.device("cuda:0")
    wl = workloads.minimax_like()
    log("minimax-like full size: cascade decode step, every sequence against the oracle")
    desc, codes, scales = gpu_cache(uq, wl, dev)
    kn, vn = new_tokens(wl, 54321)
    pre = uq.SharedPrefix(torch.as_tensor(wl.prefix_pages.astype(np.int32), device=dev),
                          torch.as_tensor(wl.prefix_lens(), device=dev), wl.shared_prefix_tokens)
    out = uq.decode_cascade(desc, wl.q.to(dev), codes, scales, torch.as_tensor(wl.page_table, device=dev),
                            torch.as_tensor(wl.context_lens, device=dev), wl.max_context, pre, 1 / math.sqrt(128), 0,
                            k_new=kn.to(dev), v_new=vn.to(dev))
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    del codes, scales
    torch.cuda.empty_cache()
    check(out, oracle_outputs(wl, dev, new=(kn, vn)), "minimax cascade step, 64 sequences")
