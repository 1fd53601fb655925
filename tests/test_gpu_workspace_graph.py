"""The decode workspace's contents on entry, and the calls under HIP graph
capture.

  * uq_decode_attention with a workspace full of garbage (every byte 0xFF,
    then random bytes) gives the output of a call on a zeroed workspace bit
    for bit, and the oracle's within max-abs 2e-3 and relative L2 1e-3
    (Algorithm 1, Decode): every partial the merge reads is written by the
    same call first.  Block grid, wave grid, head sizes 64 (one-head and
    two-head blocks) and 256, and the FP8 and BF16 comparison caches;
  * uq_decode_attention and uq_decode_step captured once in a HIP graph and
    replayed four times with new queries: every replay equals the eager call
    on the same inputs, with eager calls on the same workspace between the
    replays.  The calls enqueue kernels only (no memset, no allocation).
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads
from test_gpu_ref_caches import check_attention, gpu_cache, reference

pytestmark = pytest.mark.gpu

EDGES = [0, 1, 15, 16, 17, 31, 32, 33, 63, 64, 65, 127, 128, 129, 255, 256, 257, 500, 1000, 1023, 1024, 1025]


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def log(msg):
    print(msg, flush=True)


def contexts(seed, n, top):
    rng = np.random.default_rng(seed)
    ctx = [c for c in EDGES if c <= top][:n]
    ctx += [int(x) for x in rng.integers(1, top + 1, n - len(ctx))]
    return [int(c) for c in rng.permutation(ctx)]


def fp4_cache(uq, wl, dev):
    d = wl.head_dim
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v, head_dim=d)
    codes, scales = desc.alloc_pools(dev, fill=0xA5)
    pools = oracle.alloc_pools(wl.num_pages, wl.num_kv_heads, fill=0xA5, head_dim=d)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        slots = wl.slots(key, lo, hi, row)
        uq.quantize_kv(desc, k, v, torch.as_tensor(slots, device=dev), codes, scales)
        oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), slots, wl.num_pages, rotate_v=wl.rotate_v, pools=pools)
    torch.cuda.synchronize()
    return desc, codes, scales, pools


def garbage(ws, kind, seed):
    if kind == "zero":
        ws.zero_()
    elif kind == "ff":
        ws.fill_(0xFF)
    else:
        g = torch.Generator(device=ws.device).manual_seed(seed)
        ws.copy_(torch.randint(0, 256, ws.shape, generator=g, device=ws.device, dtype=torch.int32).to(torch.uint8))


@pytest.mark.parametrize("part,grid", [(64, "block"), (32, "wave"), (1024, "block")])
def test_fp4_garbage_workspace(uq, part, grid):
    dev = torch.device("cuda:0")
    # 40 sequences x 4 kv heads: 32-token partitions of contexts up to 2048
    # take the wave grid (2560 blocks), 64-token ones the block grid
    wl = workloads.custom(40, 64, 4, contexts(71, 40, 2048), seed=71, paging="random")
    desc, codes, scales, pools = fp4_cache(uq, wl, dev)
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    scale = 1 / math.sqrt(128)
    ws = uq.alloc_workspace(desc, wl.batch, wl.num_q_heads, wl.max_context, part, dev)
    outs = {}
    for i, kind in enumerate(("zero", "ff", "random")):
        garbage(ws, kind, i)
        outs[kind] = uq.decode_attention(desc, q, codes, scales, pt, ctx, wl.max_context, scale, part, workspace=ws)
    torch.cuda.synchronize()
    log(f"fp4 {grid} grid, partition {part}")
    assert torch.equal(outs["ff"], outs["zero"]) and torch.equal(outs["random"], outs["zero"])
    ref = oracle.decode_attention(wl.q.float().numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads,
                                  scale, wl.rotate_v)
    check_attention(outs["random"].cpu().numpy(), ref, f"fp4 {grid} grid", "exact")


@pytest.mark.parametrize("d,hq,hkv", [(64, 8, 2), (64, 12, 1), (256, 8, 2)])
def test_head_sizes_garbage_workspace(uq, d, hq, hkv):
    dev = torch.device("cuda:0")
    wl = workloads.custom(20, hq, hkv, contexts(72, 20, 700), seed=72, paging="random", head_dim=d)
    desc, codes, scales, pools = fp4_cache(uq, wl, dev)
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    scale = 1 / math.sqrt(d)
    part = 64
    ws = uq.alloc_workspace(desc, wl.batch, wl.num_q_heads, wl.max_context, part, dev)
    outs = {}
    for i, kind in enumerate(("zero", "ff")):
        garbage(ws, kind, i)
        outs[kind] = uq.decode_attention(desc, q, codes, scales, pt, ctx, wl.max_context, scale, part, workspace=ws)
    torch.cuda.synchronize()
    log(f"head size {d}, {hq} query heads, {hkv} kv heads")
    assert torch.equal(outs["ff"], outs["zero"])
    ref = oracle.decode_attention(wl.q.float().numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads,
                                  scale, wl.rotate_v)
    check_attention(outs["ff"].cpu().numpy(), ref, f"head size {d}", "exact")


@pytest.mark.parametrize("fmt", ["fp8", "bf16"])
@pytest.mark.parametrize("part", [64, 32])
def test_ref_caches_garbage_workspace(uq, fmt, part):
    dev = torch.device("cuda:0")
    wl = workloads.custom(40, 64, 4, contexts(73, 40, 2048), seed=73, paging="random")
    desc, cache = gpu_cache(uq, fmt, wl, dev)
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    scale = 1 / math.sqrt(128)
    ws = uq.ref_alloc_workspace(desc, wl.batch, wl.num_q_heads, wl.max_context, part, dev)
    outs = {}
    for i, kind in enumerate(("zero", "random")):
        garbage(ws, kind, i)
        outs[kind] = uq.ref_decode_attention(desc, q, cache, pt, ctx, wl.max_context, scale, part, workspace=ws)
    torch.cuda.synchronize()
    log(f"{fmt} partition {part}")
    assert torch.equal(outs["random"], outs["zero"])
    check_attention(outs["random"].cpu().numpy(), reference(fmt, wl, range(wl.batch), dev), f"{fmt}", fmt)


@pytest.mark.parametrize("call", ["attention", "step"])
def test_graph_replays(uq, call):
    dev = torch.device("cuda:0")
    wl = workloads.custom(40, 64, 4, contexts(74, 40, 2048), seed=74, paging="random")
    desc, codes, scales, _ = fp4_cache(uq, wl, dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    scale = 1 / math.sqrt(128)
    part = 64
    q = wl.q.to(dev).clone()
    g = torch.Generator(device=dev).manual_seed(9)
    k_new = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g, device=dev)
    v_new = torch.randn((wl.batch, wl.num_kv_heads, 128), generator=g, device=dev)
    ws = uq.alloc_workspace(desc, wl.batch, wl.num_q_heads, wl.max_context, part, dev)
    out = torch.empty((wl.batch, wl.num_q_heads, 128), dtype=torch.float32, device=dev)

    def run(o):
        if call == "attention":
            uq.decode_attention(desc, q, codes, scales, pt, ctx, wl.max_context, scale, part, workspace=ws, out=o)
        else:
            # the same new token rewritten at the same position: the step is idempotent
            uq.decode_step(desc, q, k_new, v_new, codes, scales, pt, ctx, wl.max_context, scale, part, ws, o)

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        run(out)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        run(out)
    torch.cuda.synchronize()
    want = torch.empty_like(out)
    for rep in range(4):
        q.copy_(torch.randn(q.shape, generator=g, device=dev))
        graph.replay()
        torch.cuda.synchronize()
        got = out.clone()
        run(want)   # eager, same workspace
        torch.cuda.synchronize()
        log(f"{call} replay {rep}: max-abs difference {float((got - want).abs().max()):.3e}")
        assert torch.equal(got, want), rep
