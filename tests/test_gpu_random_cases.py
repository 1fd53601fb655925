"""Seeded random combinations of the call parameters against the oracle:
head size, KV heads, group size, ragged contexts (with empty ones), paging,
partition, query and row dtypes, rotate_v, a padding row in each write.  Each case prints
its parameters before it runs.  Codes and scale bytes must match bit for
bit, attention within max-abs 2e-3 and relative L2 1e-3."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu

CASES = 64


def params(i):
    rng = np.random.default_rng(1000 + i)
    d = int(rng.choice([64, 128, 256]))
    hkv = int(rng.integers(1, 5))
    g = int(rng.choice([1, 2, 3, 6, 8, 11, 16]))
    b = int(rng.integers(1, 5))
    ctx = [int(rng.choice([0, 1, 15, 16, 17, 31, 32, 33])) if rng.random() < 0.3 else int(rng.integers(1, 1500))
           for _ in range(b)]
    if max(ctx) == 0:
        ctx[0] = 5
    part = int(rng.choice([0, 16, 32, 48, 64, 96, 256, 1024]))
    q_dt = [torch.float32, torch.bfloat16, torch.float16][int(rng.integers(0, 3))]
    row_dt = [torch.float32, torch.bfloat16, torch.float16][int(rng.integers(0, 3))]
    paging = "identity" if rng.random() < 0.3 else "random"
    rotate_v = bool(rng.random() < 0.7)
    return dict(d=d, hkv=hkv, g=g, b=b, ctx=ctx, part=part, q_dt=q_dt, row_dt=row_dt, paging=paging,
                rotate_v=rotate_v, seed=2000 + i)


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


@pytest.mark.parametrize("i", range(CASES))
def test_random_case(uq, i):
    c = params(i)
    print(f"case {i}: {c}", flush=True)
    dev = torch.device("cuda:0")
    wl = workloads.custom(c["b"], c["g"] * c["hkv"], c["hkv"], c["ctx"], seed=c["seed"], paging=c["paging"],
                          rotate_v=c["rotate_v"], head_dim=c["d"])
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v, head_dim=c["d"])
    codes, scales = desc.alloc_pools(dev, fill=0xC3)
    pools = oracle.alloc_pools(wl.num_pages, wl.num_kv_heads, fill=0xC3, head_dim=c["d"])
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev, dtype=c["row_dt"])
        slots = wl.slots(key, lo, hi, row)
        if len(slots) > 2:
            # a padding row (slot -1, written nowhere) in the middle of the batch
            m = len(slots) // 2
            k = torch.cat([k[:m], k[m:m + 1] * 3, k[m:]])
            v = torch.cat([v[:m], v[m:m + 1] * 3, v[m:]])
            slots = np.insert(slots, m, -1)
        uq.quantize_kv(desc, k, v, torch.as_tensor(slots, device=dev), codes, scales)
        oracle.quantize_kv(k.float().cpu().numpy(), v.float().cpu().numpy(), slots, wl.num_pages,
                           rotate_v=wl.rotate_v, pools=pools)
    torch.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy(), pools[0]), "codes differ"
    assert np.array_equal(scales.cpu().numpy(), pools[1]), "scale bytes differ"
    q = wl.q.to(c["q_dt"])
    out = uq.decode_attention(desc, q.to(dev), codes, scales, torch.as_tensor(wl.page_table, device=dev),
                              torch.as_tensor(wl.context_lens, device=dev), wl.max_context,
                              1 / math.sqrt(c["d"]), c["part"])
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref = oracle.decode_attention(q.float().numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads,
                                  1 / math.sqrt(c["d"]), wl.rotate_v)
    for bi, n in enumerate(c["ctx"]):
        if n == 0:
            assert np.all(got[bi] == 0)
    err = np.abs(got - ref).max()
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    print(f"case {i}: max-abs {err:.2e} rel-L2 {rel:.2e}", flush=True)
    assert np.all(np.isfinite(got))
    assert err <= 2e-3 and rel <= 1e-3
