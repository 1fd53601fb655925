"""Seeded random cascade-decode cases (uq_decode_cascade and its fused
decode step) against the oracle: shared prefixes of 1 to 12 pages, contexts
drawn around the prefix length (empty, inside the prefix with a private last
page, at page edges, equal, one longer, much longer), group sizes 1 to 16
(not only powers of two), 1 to 4 KV heads, context and prefix partitions,
query dtypes, rotate_v.  Each case prints its parameters first.

  * cascade attention: max-abs 2e-3 and relative L2 1e-3 against the fp64
    oracle, and within 2e-4 of the non-cascade call on the same pools;
  * the fused step (the new token written by the cascade call) gives pools
    and outputs identical to a separate write followed by the cascade call.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu

CASES = 32
SCALE = 1 / math.sqrt(128)


def params(i):
    rng = np.random.default_rng(5000 + i)
    hkv = int(rng.integers(1, 5))
    g = int(rng.choice([1, 2, 3, 6, 8, 11, 16]))
    b = int(rng.integers(1, 7))
    pre = 16 * int(rng.integers(1, 13))
    choices = [0, 1, max(1, pre - 15), pre - 1 if pre > 1 else 1, pre, pre + 1, pre + 16, pre + 17]
    ctx = [int(rng.choice(choices)) if rng.random() < 0.6 else pre + int(rng.integers(1, 700)) for _ in range(b)]
    if max(ctx) == 0:
        ctx[0] = pre + 3
    part = int(rng.choice([0, 32, 64, 96, 256]))
    ppart = int(rng.choice([0, 32, 64, 160]))
    q_dt = [torch.float32, torch.bfloat16, torch.float16][int(rng.integers(0, 3))]
    rotate_v = bool(rng.random() < 0.7)
    return dict(hkv=hkv, g=g, b=b, pre=pre, ctx=ctx, part=part, ppart=ppart, q_dt=q_dt, rotate_v=rotate_v,
                seed=6000 + i)


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def fill(uq, wl, dev):
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v)
    codes, scales = desc.alloc_pools(dev, fill=0x5A)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
    return desc, codes, scales


@pytest.mark.parametrize("i", range(CASES))
def test_random_cascade(uq, i):
    c = params(i)
    print(f"cascade case {i}: {c}", flush=True)
    dev = torch.device("cuda:0")
    wl = workloads.custom(c["b"], c["g"] * c["hkv"], c["hkv"], c["ctx"], seed=c["seed"], paging="random",
                          shared_prefix_tokens=c["pre"], rotate_v=c["rotate_v"])
    q = wl.q.to(c["q_dt"])
    qd = q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    prefix = uq.SharedPrefix(torch.as_tensor(wl.prefix_pages.astype(np.int32), device=dev),
                             torch.as_tensor(wl.prefix_lens(), device=dev), wl.shared_prefix_tokens, c["ppart"])

    # cascade attention against the oracle and the plain call
    desc, codes, scales = fill(uq, wl, dev)
    out = uq.decode_cascade(desc, qd, codes, scales, pt, ctx, wl.max_context, prefix, SCALE, c["part"])
    plain = uq.decode_attention(desc, qd, codes, scales, pt, ctx, wl.max_context, SCALE, c["part"])
    torch.cuda.synchronize()
    pools = oracle.alloc_pools(wl.num_pages, wl.num_kv_heads, fill=0x5A)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)   # the rows the GPU cache holds (device generator)
        oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), wl.slots(key, lo, hi, row), wl.num_pages,
                           rotate_v=wl.rotate_v, pools=pools)
    assert np.array_equal(codes.cpu().numpy(), pools[0]) and np.array_equal(scales.cpu().numpy(), pools[1])
    ref = oracle.decode_attention(q.float().numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads,
                                  SCALE, wl.rotate_v)
    got = out.cpu().numpy().astype(np.float64)
    assert np.all(np.isfinite(got))
    for bi, n in enumerate(c["ctx"]):
        if n == 0:
            assert np.all(got[bi] == 0)
    err = np.abs(got - ref).max()
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    diff = np.abs(got - plain.cpu().numpy()).max()
    print(f"cascade case {i}: max-abs {err:.2e} rel-L2 {rel:.2e}, vs plain {diff:.2e}", flush=True)
    assert err <= 2e-3 and rel <= 1e-3
    assert diff <= 5e-4

    # the fused step against a separate write + cascade call
    g = torch.Generator(device=dev).manual_seed(c["seed"])
    k_new = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g, device=dev)
    v_new = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g, device=dev)
    n = wl.context_lens.astype(np.int64)
    last = np.maximum(n - 1, 0)
    slots = wl.page_table[np.arange(wl.batch), last // 16].astype(np.int64) * 16 + last % 16
    slots = torch.as_tensor(np.where(n > 0, slots, -1), device=dev)
    results = []
    for fused in (False, True):
        desc, codes, scales = fill(uq, wl, dev)
        if not fused:
            uq.quantize_kv(desc, k_new, v_new, slots, codes, scales)
        o = uq.decode_cascade(desc, qd, codes, scales, pt, ctx, wl.max_context, prefix, SCALE, c["part"],
                              k_new=k_new if fused else None, v_new=v_new if fused else None)
        torch.cuda.synchronize()
        results.append((codes.cpu(), scales.cpu(), o.cpu()))
    for a, b in zip(*results):
        assert torch.equal(a, b), f"case {i}: fused step differs from write + cascade"
