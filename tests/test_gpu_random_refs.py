"""Seeded random cases for the comparison caches (FP8 E4M3 with per-tensor
scales, BF16, Ultra-TQ) through uq_ref_*: 1 to 4 KV heads, group sizes 1
to 16 (not only powers of two), ragged contexts with empty ones and page
edges, partitions, f32/bf16 queries and f32/bf16/f16 rows, FP8 scales.
Attention against the same CPU references as the fixed cases (plain
PyTorch over the dequantized cache for FP8 and BF16, the oracle for
Ultra-TQ), and the fused step against a separate write + decode, bit for
bit.  Each case prints its parameters first."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads
from paper_2606_20474_amd.codebook import default_tq_codebook
from test_gpu_ref_caches import MAX_ABS, REL_L2, attention, query_values, seq_values

pytestmark = pytest.mark.gpu

SCALE = 1 / math.sqrt(128)
CASES = 16


def params(fmt, i):
    rng = np.random.default_rng({"fp8": 9100, "bf16": 9200, "tq4": 9300}[fmt] + i)
    hkv = int(rng.integers(1, 5))
    g = int(rng.choice([1, 2, 3, 6, 8, 11, 16]))
    b = int(rng.integers(1, 5))
    ctx = [int(rng.choice([0, 1, 15, 16, 17, 31, 32, 33])) if rng.random() < 0.3 else int(rng.integers(1, 1200))
           for _ in range(b)]
    if max(ctx) == 0:
        ctx[0] = 7
    part = int(rng.choice([0, 32, 64, 96, 256]))
    q_dt = [torch.float32, torch.bfloat16][int(rng.integers(0, 2))]
    row_dt = [torch.float32, torch.bfloat16, torch.float16][int(rng.integers(0, 3))]
    ks, vs = (float(rng.choice([0.05, 0.3, 1.0])), float(rng.choice([0.05, 0.3, 1.0]))) if fmt == "fp8" else (1.0, 1.0)
    return dict(hkv=hkv, g=g, b=b, ctx=ctx, part=part, q_dt=q_dt, row_dt=row_dt, ks=ks, vs=vs,
                seed={"fp8": 9500, "bf16": 9600, "tq4": 9700}[fmt] + i)


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def fill(uq, fmt, wl, dev, c):
    desc = uq.RefCacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, fmt=fmt, k_scale=c["ks"],
                           v_scale=c["vs"])
    cache = desc.alloc_cache(dev, fill=0x5A)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev, dtype=c["row_dt"])
        uq.ref_write_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), cache)
    return desc, cache


@pytest.mark.parametrize("fmt", ["fp8", "bf16", "tq4"])
@pytest.mark.parametrize("i", range(CASES))
def test_random_ref_cache(uq, fmt, i):
    c = params(fmt, i)
    print(f"{fmt} case {i}: {c}", flush=True)
    dev = torch.device("cuda:0")
    wl = workloads.custom(c["b"], c["g"] * c["hkv"], c["hkv"], c["ctx"], seed=c["seed"], paging="random")
    q = wl.q.to(c["q_dt"])
    qd = q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)

    desc, cache = fill(uq, fmt, wl, dev, c)
    out = uq.ref_decode_attention(desc, qd, cache, pt, ctx, wl.max_context, SCALE, c["part"])
    torch.cuda.synchronize()
    got = out.cpu().numpy().astype(np.float64)
    if fmt == "tq4":
        cb = default_tq_codebook(128)
        pools = oracle.tq4_alloc_cache(wl.num_pages, wl.num_kv_heads, fill=0x5A)
        for key, lo, hi, row in wl.segments():
            k, v = wl.kv(key, lo, hi, device=dev, dtype=c["row_dt"])
            oracle.tq4_write(k.float().cpu().numpy(), v.float().cpu().numpy(), wl.slots(key, lo, hi, row),
                             wl.num_pages, cb, pools)
        assert np.array_equal(cache.cpu().numpy(), pools), "cache bytes differ"
        ref = oracle.tq4_decode_attention(q.float().numpy(), pools, wl.page_table, wl.context_lens,
                                          wl.num_kv_heads, cb)
        max_abs, rel_l2 = 2e-3, 1e-3
    else:
        ref = np.zeros_like(got)
        for b in range(wl.batch):
            kd, vd = seq_values(fmt, wl, b, dev, c["ks"], c["vs"], in_dtype=c["row_dt"])
            ref[b] = attention(query_values(fmt, q[b]), kd, vd, wl.group)
        max_abs, rel_l2 = MAX_ABS[fmt], REL_L2[fmt]
    assert np.all(np.isfinite(got))
    for b, n in enumerate(c["ctx"]):
        if n == 0:
            assert np.all(got[b] == 0)
    err = np.abs(got - ref).max()
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    print(f"{fmt} case {i}: max-abs {err:.2e} rel-L2 {rel:.2e}", flush=True)
    assert err <= max_abs and rel <= rel_l2

    # fused step against write + decode
    g = torch.Generator(device=dev).manual_seed(c["seed"])
    k_new = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g, device=dev).to(c["row_dt"])
    v_new = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g, device=dev).to(c["row_dt"])
    n = wl.context_lens.astype(np.int64)
    last = np.maximum(n - 1, 0)
    slots = wl.page_table[np.arange(wl.batch), last // 16].astype(np.int64) * 16 + last % 16
    slots = torch.as_tensor(np.where(n > 0, slots, -1), device=dev)
    results = []
    for fused in (False, True):
        desc, cache = fill(uq, fmt, wl, dev, c)
        if fused:
            o = uq.ref_decode_step(desc, qd, k_new, v_new, cache, pt, ctx, wl.max_context, SCALE, c["part"])
        else:
            uq.ref_write_kv(desc, k_new, v_new, slots, cache)
            o = uq.ref_decode_attention(desc, qd, cache, pt, ctx, wl.max_context, SCALE, c["part"])
        torch.cuda.synchronize()
        results.append((cache.cpu(), o.cpu()))
    assert torch.equal(results[0][0], results[1][0]), f"{fmt} case {i}: caches differ"
    assert torch.equal(results[0][1], results[1][1]), f"{fmt} case {i}: outputs differ"
