"""The one-wave-per-partition grid of the partition launch.

A launch with at least 8 blocks per CU of W consecutive partitions each (W =
8 waves per block for the FP4 and FP8 caches where that many blocks of 8
exist, else 4; 4 for Ultra-TQ, 2 for BF16), head size 128 and no shared
prefix gives every wave one whole partition: the wave streams it through
its own ring, the block merges its W partials and the merge kernel finishes
every row, also the rows of contexts that fit one partition.  The shapes
here (40 sequences, 4 kv heads, 16-token partitions of contexts up to 2048
tokens: 40 x 4 x 16 = 2560 blocks of 8) take that grid while the oracle
still finishes them in seconds; 32-token partitions take it with blocks of
4 (40 x 4 x 16 = 2560 blocks), 64-token partitions of the same data (1280
blocks of 4) the block-per-partition grid.
  * the page-gather probe fills exactly the wave grid's sink words, and reads
    the same bytes as on the block grid;
  * FP4 decode against the oracle (Algorithm 1, Decode; max-abs 2e-3,
    relative L2 1e-3) for both V modes, ragged contexts at page, stage and
    partition edges, an empty context;
  * the fused step (new token written at the last position) leaves the pools
    and the output bit for bit as the write followed by the attention, for
    the four cache formats, and its partials-only form with the separate
    merge call gives the same output;
  * the comparison caches against their CPU expectation, and every format
    against its own block-grid output.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads
from test_gpu_ref_caches import MAX_ABS, REL_L2, check_attention, gpu_cache, reference, run
from test_gpu_step import Cache, compare_step, new_tokens

pytestmark = pytest.mark.gpu

SCALE = 1 / math.sqrt(128)
EDGES = [0, 1, 15, 16, 17, 31, 32, 33, 63, 64, 65, 95, 96, 97, 127, 128, 129, 255, 256, 257, 500, 777, 1000, 1023,
         1024, 1025, 1500, 2000, 2047, 2048]
WAVE_PART, BLOCK_PART = 16, 64


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def log(msg):
    print(msg, flush=True)


def contexts(seed):
    rng = np.random.default_rng(seed)
    ctx = EDGES + [int(x) for x in rng.integers(1, 2049, 40 - len(EDGES))]
    return [int(c) for c in rng.permutation(ctx)]


def workload(seed, rotate_v=True, hq=64):
    return workloads.custom(40, hq, 4, contexts(seed), seed=seed, paging="random", rotate_v=rotate_v)


def fp4_cache(uq, wl, dev):
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v)
    codes, scales = desc.alloc_pools(dev, fill=0xA5)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
    torch.cuda.synchronize()
    return desc, codes, scales


def oracle_out(wl, dev, q=None):
    """The oracle's own cache of the same K/V (drawn on the device, as the
    GPU cache's) and its attention."""
    pools = oracle.alloc_pools(wl.num_pages, wl.num_kv_heads)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), wl.slots(key, lo, hi, row), wl.num_pages,
                           rotate_v=wl.rotate_v, pools=pools)
    q = wl.q if q is None else q
    return oracle.decode_attention(q.float().numpy(), pools, wl.page_table, wl.context_lens, wl.num_kv_heads, SCALE,
                                   wl.rotate_v)


def check(got, ref, what):
    got = np.asarray(got, np.float64)
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    log(f"{what}: max-abs {err.max():.3e} rel-L2 {rel:.3e}")
    assert np.all(np.isfinite(got)), what
    assert err.max() <= 2e-3, (what, err.max())
    assert rel <= 1e-3, (what, rel)


def test_probe_fills_the_wave_grid(uq):
    dev = torch.device("cuda:0")
    wl = workload(61)
    desc, codes, scales = fp4_cache(uq, wl, dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    np_wave = -(-wl.max_context // WAVE_PART)
    sinks = {}
    for part in (WAVE_PART, BLOCK_PART):
        n = 4 * -(-wl.max_context // part) * wl.num_kv_heads * wl.batch   # the documented bound
        sink = torch.full((n,), -1, dtype=torch.int32, device=dev)
        uq.probe_page_gather(desc, wl.num_q_heads, codes, scales, pt, ctx, wl.max_context, part, sink)
        torch.cuda.synchronize()
        sinks[part] = sink.cpu().numpy()
    s = sinks[WAVE_PART]
    used = -(-np_wave // 8) * wl.num_kv_heads * wl.batch * 8
    log(f"wave grid: {used} of {s.size} sink words")
    assert np.all(s[:used] != -1) and np.all(s[used:] == -1)
    w = s[:used].reshape(-1, wl.batch, wl.num_kv_heads, 8)   # [partition group][sequence][kv head][wave]
    for b, c in enumerate(wl.context_lens):
        nparts = -(-int(c) // WAVE_PART)
        flat = w[:, b].transpose(0, 2, 1).reshape(-1, wl.num_kv_heads)   # [partition][kv head]
        assert np.all(flat[nparts:] == 0), b
    # every page read once on either grid (and the same padding reads)
    used_b = -(-wl.max_context // BLOCK_PART) * wl.num_kv_heads * wl.batch * 4   # blocks of 4 waves
    assert np.all(sinks[BLOCK_PART][:used_b] != -1)
    assert np.bitwise_xor.reduce(s[:used].view(np.uint32)) == np.bitwise_xor.reduce(
        sinks[BLOCK_PART][:used_b].view(np.uint32))


@pytest.mark.parametrize("rotate_v", [True, False])
def test_fp4_decode_against_oracle(uq, rotate_v):
    dev = torch.device("cuda:0")
    wl = workload(62, rotate_v=rotate_v)
    log(f"wave grid fp4 decode rotate_v={rotate_v}")
    desc, codes, scales = fp4_cache(uq, wl, dev)
    ref = oracle_out(wl, dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    outs = {}
    for part in (WAVE_PART, BLOCK_PART, 32, 48):
        out = uq.decode_attention(desc, wl.q.to(dev), codes, scales, pt, ctx, wl.max_context, SCALE, part)
        torch.cuda.synchronize()
        outs[part] = out.cpu().numpy().astype(np.float64)
        check(outs[part], ref, f"partition {part}")
    empty = [b for b, c in enumerate(wl.context_lens) if c == 0]
    assert empty and np.all(outs[WAVE_PART][empty] == 0)


def test_fp4_group_8_bf16_query(uq):
    dev = torch.device("cuda:0")
    wl = workload(63, hq=32)
    desc, codes, scales = fp4_cache(uq, wl, dev)
    q = wl.q.to(torch.bfloat16)
    ref = oracle_out(wl, dev, q)
    out = uq.decode_attention(desc, q.to(dev), codes, scales, torch.as_tensor(wl.page_table, device=dev),
                              torch.as_tensor(wl.context_lens, device=dev), wl.max_context, SCALE, WAVE_PART,
                              out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    got = out.float().cpu().numpy().astype(np.float64)
    err = np.abs(got - ref).max()
    log(f"group 8, bf16 query and output: max-abs {err:.3e}")
    assert err <= 2e-3 + np.abs(ref).max() * 2.0 ** -8


@pytest.mark.parametrize("fmt", ["fp4", "fp8", "bf16", "tq4"])
def test_step_matches_write_then_attend(uq, fmt):
    dev = torch.device("cuda:0")
    wl = workload(64)
    log(f"wave grid step {fmt}")
    out = compare_step(uq, fmt, wl, dev, WAVE_PART)
    # partials only, then the separate merge call
    c = Cache(uq, fmt, wl, dev)
    k_new, v_new = new_tokens(wl, dev)
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    if fmt == "fp4":
        ws = uq.alloc_workspace(c.desc, wl.batch, wl.num_q_heads, wl.max_context, WAVE_PART, dev)
        o2 = torch.empty_like(out)
        uq.decode_step(c.desc, q, k_new, v_new, *c.bufs, pt, ctx, wl.max_context, SCALE, WAVE_PART, ws, o2,
                       partials_only=True)
        uq.decode_merge(c.desc, wl.batch, wl.num_q_heads, ctx, wl.max_context, WAVE_PART, ws, o2)
    else:
        ws = uq.ref_alloc_workspace(c.desc, wl.batch, wl.num_q_heads, wl.max_context, WAVE_PART, dev)
        o2 = torch.empty_like(out)
        uq.ref_decode_step(c.desc, q, k_new, v_new, *c.bufs, pt, ctx, wl.max_context, SCALE, WAVE_PART, ws, o2,
                           partials_only=True)
        uq.ref_decode_merge(c.desc, wl.batch, wl.num_q_heads, ctx, wl.max_context, WAVE_PART, ws, o2)
    torch.cuda.synchronize()
    assert torch.equal(o2, out)


@pytest.mark.parametrize("fmt", ["fp8", "bf16"])
def test_ref_caches_against_cpu(uq, fmt):
    dev = torch.device("cuda:0")
    wl = workload(65)
    log(f"wave grid ref decode {fmt}")
    desc, cache = gpu_cache(uq, fmt, wl, dev)
    ref = reference(fmt, wl, range(wl.batch), dev)
    check_attention(run(uq, desc, wl, cache, dev, WAVE_PART), ref, f"{fmt} wave grid", fmt)


@pytest.mark.parametrize("fmt", ["fp4", "fp8", "bf16", "tq4"])
def test_wave_grid_against_block_grid(uq, fmt):
    """The two grids compute the same attention (each partition's partial in
    a different order): within the parity bounds of the format."""
    dev = torch.device("cuda:0")
    wl = workload(66)
    c = Cache(uq, fmt, wl, dev)
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    a = c.attend(q, pt, ctx, WAVE_PART).cpu().numpy().astype(np.float64)
    b = c.attend(q, pt, ctx, BLOCK_PART).cpu().numpy().astype(np.float64)
    torch.cuda.synchronize()
    err = np.abs(a - b).max()
    log(f"{fmt}: wave grid against block grid max-abs {err:.3e}")
    tol = {"fp4": 2e-3, "tq4": 2e-3, "bf16": MAX_ABS["bf16"], "fp8": MAX_ABS["fp8"]}[fmt]
    assert np.all(np.isfinite(a)) and err <= tol
    assert np.linalg.norm(a - b) / np.linalg.norm(b) <= {"fp8": REL_L2["fp8"]}.get(fmt, 1e-3)
