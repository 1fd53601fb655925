"""Seeded random cases on the two launch shapes that small cases never reach,
against the oracle (Algorithm 1, Decode; max-abs 2e-3, relative L2 1e-3):

  * the one-wave-per-partition grid: 32-48 sequences of ragged contexts up
    to 2048 tokens (one of exactly 2048) in 16- or 32-token partitions, so
    that the launch has at least 2048 blocks of 8 partitions (16-token
    partitions) or of 4 (32-token);
  * long partitions: 8192 or 16384 tokens per block over contexts up to
    20000, so that every wave of a block walks more than 32 page pairs and
    takes its later page ids from its LDS slot.

Group size, rotate_v and the query dtype are drawn too.  Each case prints
its parameters and the grid the launch rule gives before it runs."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu

CASES = 12
EDGES = [0, 1, 15, 16, 17, 31, 32, 33, 255, 256, 257, 2047, 2048]


def params(i):
    rng = np.random.default_rng(5000 + i)
    g = int(rng.choice([1, 2, 4, 6, 8, 11, 16]))
    q_dt = [torch.float32, torch.bfloat16, torch.float16][int(rng.integers(0, 3))]
    rotate_v = bool(rng.random() < 0.7)
    if i % 2 == 0:
        b = int(rng.integers(32, 49))
        hkv = 4
        ctx = [int(rng.choice(EDGES)) if rng.random() < 0.3 else int(rng.integers(1, 2049)) for _ in range(b)]
        ctx[int(rng.integers(0, b))] = 2048   # 16-token partitions: blocks of 8; 32-token: blocks of 4
        part = int(rng.choice([16, 32]))
    else:
        b = int(rng.integers(1, 4))
        hkv = int(rng.integers(1, 3))
        ctx = [int(rng.integers(8000, 20001)) for _ in range(b)]
        part = int(rng.choice([8192, 16384]))
    return dict(b=b, hkv=hkv, g=g, ctx=ctx, part=part, q_dt=q_dt, rotate_v=rotate_v, seed=6000 + i)


def grid_of(c):
    """The launch rule of the partition kernel (head size 128, no shared
    prefix): one wave per partition in blocks of W = 8 partitions when there
    are at least 16 partitions and that gives at least 8 blocks per CU (256
    CUs), else blocks of 4 under the same block count, else one block per
    partition."""
    np_ = -(-max(c["ctx"]) // c["part"]) if max(c["ctx"]) > 0 else 1
    for w in (8, 4):
        if np_ >= max(w, 16 if w == 8 else 0) and c["b"] * c["hkv"] * -(-np_ // w) >= 8 * 256:
            return f"wave grid, {w} partitions per block"
    return "one block per partition"


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


@pytest.mark.parametrize("i", range(CASES))
def test_random_grid_case(uq, i):
    c = params(i)
    print(f"grid case {i}: {c}; {grid_of(c)}", flush=True)
    dev = torch.device("cuda:0")
    wl = workloads.custom(c["b"], c["g"] * c["hkv"], c["hkv"], c["ctx"], seed=c["seed"], paging="random",
                          rotate_v=c["rotate_v"])
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v)
    codes, scales = desc.alloc_pools(dev, fill=0x3C)
    pools = oracle.alloc_pools(wl.num_pages, wl.num_kv_heads, fill=0x3C)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        slots = wl.slots(key, lo, hi, row)
        uq.quantize_kv(desc, k, v, torch.as_tensor(slots, device=dev), codes, scales)
        oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), slots, wl.num_pages, rotate_v=wl.rotate_v, pools=pools)
    torch.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy(), pools[0]), "codes differ"
    assert np.array_equal(scales.cpu().numpy(), pools[1]), "scale bytes differ"
    q = wl.q.to(c["q_dt"])
    out = uq.decode_attention(desc, q.to(dev), codes, scales, torch.as_tensor(wl.page_table, device=dev),
                              torch.as_tensor(wl.context_lens, device=dev), wl.max_context, 1 / math.sqrt(128),
                              c["part"])
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    ref = oracle.decode_attention(q.float().numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads,
                                  1 / math.sqrt(128), wl.rotate_v)
    empty = [bi for bi, n in enumerate(c["ctx"]) if n == 0]
    assert np.all(got[empty] == 0), "empty contexts give zeros"
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    print(f"grid case {i}: max-abs {err.max():.3e} rel-L2 {rel:.3e}", flush=True)
    assert np.all(np.isfinite(got))
    assert err.max() <= 2e-3, (i, err.max())
    assert rel <= 1e-3, (i, rel)
