"""The kernel timing hook (uq_time_next_launch): the timed launch computes
the same bytes as an untimed one, its events bracket the kernel inside the
events recorded around the call, and the setting is used once."""
import math

import numpy as np
import pytest
import torch

from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def events(stream, n=2):
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
    for e in ev:
        e.record(stream)   # creates the HIP event
    torch.cuda.synchronize()
    return ev


def test_timed_decode_matches_and_nests(uq):
    dev = torch.device("cuda:0")
    print("timing hook: decode", flush=True)
    wl = workloads.custom(4, 16, 2, [3000, 700, 1, 4096], seed=71, paging="random")
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages)
    codes, scales = desc.alloc_pools(dev)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    st = torch.cuda.current_stream()

    def run():
        return uq.decode_attention(desc, q, codes, scales, pt, ctx, wl.max_context, 1 / math.sqrt(128), 256)

    plain = run()
    outer_a, outer_b, ka, kb = events(st, 4)
    outer_a.record(st)
    uq.time_next_launch(ka, kb)
    timed = run()
    outer_b.record(st)
    torch.cuda.synchronize()
    assert torch.equal(plain, timed)
    k_ms = ka.elapsed_time(kb)
    o_ms = outer_a.elapsed_time(outer_b)
    print(f"kernel {k_ms * 1e3:.1f} us inside {o_ms * 1e3:.1f} us", flush=True)
    assert 0 < k_ms <= o_ms
    # used once: a second call leaves the pair alone
    again = run()
    torch.cuda.synchronize()
    assert torch.equal(plain, again)
    assert ka.elapsed_time(kb) == k_ms


def test_timed_quantize_matches(uq):
    dev = torch.device("cuda:0")
    print("timing hook: quantize", flush=True)
    desc = uq.CacheDesc(num_kv_heads=4, num_pages=64)
    g = torch.Generator().manual_seed(72)
    k = torch.randn((500, 4, 128), generator=g).bfloat16().to(dev)
    v = torch.randn((500, 4, 128), generator=g).bfloat16().to(dev)
    slots = torch.as_tensor(np.random.default_rng(72).permutation(64 * 16)[:500].astype(np.int64), device=dev)
    c1, s1 = desc.alloc_pools(dev, fill=0x11)
    c2, s2 = desc.alloc_pools(dev, fill=0x11)
    uq.quantize_kv(desc, k, v, slots, c1, s1)
    st = torch.cuda.current_stream()
    ka, kb = events(st)
    uq.time_next_launch(ka, kb)
    uq.quantize_kv(desc, k, v, slots, c2, s2)
    torch.cuda.synchronize()
    assert torch.equal(c1, c2) and torch.equal(s1, s2)
    assert ka.elapsed_time(kb) > 0
