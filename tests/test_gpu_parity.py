"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Codes, scale bytes and FP8 query bytes must match bit for bit.  Attention
outputs must match within max-abs 2e-3 and relative L2 1e-3 of the fp64
oracle, which quantises the same seeded K/V on its own.
"""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu

MAX_ABS = 2e-3
REL_L2 = 1e-3


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def log(msg):
    print(msg, flush=True)


def check_attention(got, ref, what):
    got = np.asarray(got, np.float64)
    ref = np.asarray(ref, np.float64)
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    log(f"{what}: max-abs {err.max():.3e} rel-L2 {rel:.3e}")
    assert np.all(np.isfinite(got)), what
    assert err.max() <= MAX_ABS, (what, err.max())
    assert rel <= REL_L2, (what, rel)


def gpu_cache(uq, wl, device, fill=0xA5, in_dtype=torch.float32):
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v)
    codes, scales = desc.alloc_pools(device, fill=fill)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=device, dtype=in_dtype)
        slots = torch.as_tensor(wl.slots(key, lo, hi, row), device=device)
        uq.quantize_kv(desc, k, v, slots, codes, scales)
    torch.cuda.synchronize()
    return desc, codes, scales


def oracle_cache(wl, seqs, device, in_dtype=torch.float32):
    """Oracle pools for the sequences `seqs` only, in a compact page pool
    (page ids renumbered; attention does not depend on the numbering)."""
    maxp = wl.max_pages_per_seq
    pt = np.arange(len(seqs) * maxp, dtype=np.int32).reshape(len(seqs), maxp)
    pools = oracle.alloc_pools(len(seqs) * maxp, wl.num_kv_heads)
    for i, b in enumerate(seqs):
        for key, lo, hi in wl.sequence_segments(b):
            k, v = wl.kv(key, lo, hi, device=device, dtype=in_dtype)
            k = k.float().cpu().numpy()
            v = v.float().cpu().numpy()
            pos = np.arange(lo, hi, dtype=np.int64)
            slots = pt[i, pos // 16].astype(np.int64) * 16 + pos % 16
            oracle.quantize_kv(k, v, slots, len(seqs) * maxp, rotate_v=wl.rotate_v, pools=pools)
    return pools, pt


def run_decode(uq, wl, desc, codes, scales, device, partition=None, q=None, out_dtype=torch.float32, q_dtype=None):
    q = (wl.q if q is None else q).to(device)
    pt = torch.as_tensor(wl.page_table, device=device)
    ctx = torch.as_tensor(wl.context_lens, device=device)
    part = wl.partition_tokens if partition is None else partition
    out = uq.decode_attention(desc, q, codes, scales, pt, ctx, wl.max_context, 1 / math.sqrt(128), part,
                              out_dtype=out_dtype, q_dtype=q_dtype)
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


# --------------------------------------------------------------------------
# quantize-on-write: bit-exact codes and scale bytes
# --------------------------------------------------------------------------
def test_quantize_tiny_bit_exact(uq):
    dev = torch.device("cuda:0")
    wl = workloads.tiny()
    log("quantize tiny: fp32 4096 tokens")
    desc, codes, scales = gpu_cache(uq, wl, dev)
    pools = oracle.alloc_pools(wl.num_pages, 1, fill=0xA5)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), wl.slots(key, lo, hi, row), wl.num_pages, pools=pools)
    assert np.array_equal(codes.cpu().numpy(), pools[0])
    assert np.array_equal(scales.cpu().numpy(), pools[1])


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16, torch.float16])
@pytest.mark.parametrize("rotate_v", [True, False])
def test_quantize_dtypes_ragged_bit_exact(uq, dtype, rotate_v):
    dev = torch.device("cuda:0")
    log(f"quantize ragged dtype={dtype} rotate_v={rotate_v}")
    Hkv, T, num_pages = 3, 1001, 80
    g = torch.Generator(device=dev).manual_seed(11)
    k = (torch.randn((T, Hkv, 128), generator=g, device=dev) * 3).to(dtype)
    v = (torch.randn((T, Hkv, 128), generator=g, device=dev) * 0.01).to(dtype)
    k[:7] = 0          # all-zero groups -> scale byte 0
    k[7, 0, :] = -0.0
    v[9, 1, 5] = 1e4   # one huge value in a group
    perm = torch.randperm(num_pages * 16, generator=torch.Generator().manual_seed(5))[:T].numpy().astype(np.int64)
    perm[3] = -1                     # padding token
    perm[4] = num_pages * 16 + 7     # outside the pool: skipped
    desc = uq.CacheDesc(num_kv_heads=Hkv, num_pages=num_pages, rotate_v=rotate_v)
    codes, scales = desc.alloc_pools(dev, fill=0x5A)
    uq.quantize_kv(desc, k, v, torch.as_tensor(perm, device=dev), codes, scales)
    torch.cuda.synchronize()
    pools = oracle.alloc_pools(num_pages, Hkv, fill=0x5A)
    oracle.quantize_kv(k.float().cpu().numpy(), v.float().cpu().numpy(), perm, num_pages, rotate_v=rotate_v,
                       pools=pools)
    assert np.array_equal(codes.cpu().numpy(), pools[0])
    assert np.array_equal(scales.cpu().numpy(), pools[1])


def test_quantize_strided_rows(uq):
    """K and V as views into a fused [T, (Hq + 2 Hkv) * 128] projection output."""
    dev = torch.device("cuda:0")
    Hq, Hkv, T = 4, 2, 96
    g = torch.Generator(device=dev).manual_seed(3)
    qkv = torch.randn((T, (Hq + 2 * Hkv) * 128), generator=g, device=dev).bfloat16()
    k = qkv[:, Hq * 128:(Hq + Hkv) * 128].view(T, Hkv, 128)
    v = qkv[:, (Hq + Hkv) * 128:].view(T, Hkv, 128)
    slots = torch.arange(T, device=dev, dtype=torch.int64) + 16
    desc = uq.CacheDesc(num_kv_heads=Hkv, num_pages=8)
    codes, scales = desc.alloc_pools(dev, fill=0)
    uq.quantize_kv(desc, k, v, slots, codes, scales, token_stride=qkv.stride(0))
    torch.cuda.synchronize()
    pools = oracle.quantize_kv(k.float().cpu().numpy(), v.float().cpu().numpy(), slots.cpu().numpy(), 8)
    assert np.array_equal(codes.cpu().numpy(), pools[0]) and np.array_equal(scales.cpu().numpy(), pools[1])


def test_quantize_write_workload_bit_exact(uq):
    """65536-token bf16 prefill into random pages + a 1-token append for 256
    sequences through a page table (logical slots); every pool byte checked."""
    dev = torch.device("cuda:0")
    ww = workloads.WriteWorkload()
    log("quantize write workload: 65536 x 8 heads bf16 + 256 appends")
    data = ww.build(device=dev)
    kp, vp, pslots = data["prefill"]
    ka, va, aslots, pt, ctx = data["append"]
    desc = uq.CacheDesc(num_kv_heads=ww.num_kv_heads, num_pages=ww.num_pages)
    codes, scales = desc.alloc_pools(dev, fill=0xA5)
    uq.quantize_kv(desc, kp, vp, torch.as_tensor(pslots, device=dev), codes, scales)
    uq.quantize_kv(desc, ka, va, torch.as_tensor(aslots, device=dev), codes, scales,
                   page_table=torch.as_tensor(pt, device=dev))
    torch.cuda.synchronize()
    pools = oracle.alloc_pools(ww.num_pages, ww.num_kv_heads, fill=0xA5)
    oracle.quantize_kv(kp.float().cpu().numpy(), vp.float().cpu().numpy(), pslots, ww.num_pages, pools=pools)
    phys = pt[np.arange(ww.append_seqs), ctx // 16].astype(np.int64) * 16 + ctx % 16
    oracle.quantize_kv(ka.float().cpu().numpy(), va.float().cpu().numpy(), phys, ww.num_pages, pools=pools)
    assert np.array_equal(codes.cpu().numpy(), pools[0])
    assert np.array_equal(scales.cpu().numpy(), pools[1])


def test_prepare_query_bit_exact(uq):
    dev = torch.device("cuda:0")
    g = torch.Generator().manual_seed(9)
    q = torch.randn((300, 128), generator=g) * torch.logspace(-4, 3, 300).unsqueeze(1)
    q[0] = 0
    q[1] = -0.0
    q[2, 0] = 1e6   # saturates after the rotation
    desc = uq.CacheDesc(num_kv_heads=1, num_pages=1)
    for dt in (torch.float32, torch.bfloat16, torch.float16):
        qd = q.to(dt)
        got = uq.prepare_query(desc, qd.to(dev)).cpu().numpy()
        ref = oracle.prepare_query(qd.float().numpy())
        assert np.array_equal(got, ref), dt


@pytest.mark.parametrize("d", [64, 128, 256])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_write_e2m1_ties_go_to_even_code(uq, d, dtype):
    """V rows (rotate_v off, so V is encoded as given) whose groups hold
    every E2M1 midpoint of the scaled grid: each group's first channel is
    6 * 2^k, which sets E = k (fl32(0.156 * 6) rounds to exponent 0); the
    others are +-{0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5} * 2^k, both zeros,
    exact levels and values past 6 (at most 9, so that the group maximum
    keeps E = k).  Every pool byte against the oracle."""
    dev = torch.device("cuda:0")
    ties = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]
    group = [6.0] + ties + [-t for t in ties] + [0.0, -0.0, 0.5, -0.5, -1.5, 4.0, -6.0, 7.5, -9.0, 3.0, -2.0, 1.0,
                                                 0.2499, 0.7501, -5.0001, 4.9999, 2.0]
    assert len(group) == 32
    rows = []
    for k in (-30, -8, 0, 7, 40):
        for rot in range(4):   # the values move between channels, the anchor between groups
            g = np.roll(np.array(group, np.float64) * 2.0 ** k, rot * 5)
            rows.append(np.concatenate([np.roll(g, 3 * j) for j in range(d // 32)]))
    v = np.stack(rows).astype(np.float32)
    assert np.all(np.isfinite(v))
    T = len(v)
    kv = torch.as_tensor(v).reshape(T, 1, d).to(dtype)
    slots = np.arange(T, dtype=np.int64)
    pages = (T + 15) // 16
    desc = uq.CacheDesc(num_kv_heads=1, num_pages=pages, rotate_v=False, head_dim=d)
    codes, scales = desc.alloc_pools(dev, fill=0x77)
    uq.quantize_kv(desc, kv.to(dev), kv.to(dev), torch.as_tensor(slots, device=dev), codes, scales)
    pools = oracle.alloc_pools(pages, 1, fill=0x77, head_dim=d)
    oracle.quantize_kv(kv.float().numpy(), kv.float().numpy(), slots, pages, rotate_v=False, pools=pools)
    assert np.array_equal(scales.cpu().numpy(), pools[1])
    assert np.array_equal(codes.cpu().numpy(), pools[0])


def e4m3_tie_rows():
    """Query rows c * e_j whose rotation lands every channel on an exact
    midpoint between two adjacent E4M3 values: the butterfly of c e_j is
    +-c in every channel (additions of zeros are exact), then one fp32
    multiply by fl32(1/sqrt(128)), so c is chosen with fl32(c * r) equal to
    the midpoint.  One row per midpoint and sign, j varied so that the
    Hadamard row's signs vary too.  Such a c exists for 96 of the 126
    midpoints: where c = m / r has the larger exponent, consecutive products
    fl32(c * r) lie about 1.4 ulp of m apart and can step over m."""
    r = np.float32(1.0 / math.sqrt(128.0))
    rows = []
    for b in range(0x7E):
        m = np.float32((oracle.e4m3_value(b) + oracle.e4m3_value(b + 1)) / 2)
        c0 = np.float32(float(m) / float(r))
        cands = [c0]
        up = down = c0
        for _ in range(8):
            up = np.nextafter(up, np.float32(np.inf))
            down = np.nextafter(down, np.float32(-np.inf))
            cands += [up, down]
        for c in cands:
            if np.float32(c * r) == m:
                for sign in (1, -1):
                    row = np.zeros(128, np.float32)
                    row[(b * 7 + (sign > 0)) % 128] = sign * c
                    rows.append(row)
                break
    return np.stack(rows)


def test_prepare_query_ties_go_to_even_code(uq):
    q = e4m3_tie_rows()
    assert len(q) == 2 * 96, len(q)
    log(f"prepare_query: {len(q)} rows on exact E4M3 midpoints")
    desc = uq.CacheDesc(num_kv_heads=1, num_pages=1)
    got = uq.prepare_query(desc, torch.as_tensor(q, device=torch.device("cuda:0"))).cpu().numpy()
    ref = oracle.prepare_query(q)
    assert np.array_equal(got, ref)
    assert np.all((got & 0x7F) % 2 == 0), "a tie rounded to an odd code"


# --------------------------------------------------------------------------
# decode attention
# --------------------------------------------------------------------------
@pytest.fixture(scope="module")
def tiny_case(uq):
    dev = torch.device("cuda:0")
    wl = workloads.tiny()
    desc, codes, scales = gpu_cache(uq, wl, dev)
    pools, pt = oracle_cache(wl, [0], dev)
    ref = oracle.decode_attention(wl.q.numpy(), pools, pt, wl.context_lens, 1, 1 / math.sqrt(128), True)
    return wl, desc, codes, scales, ref


@pytest.mark.parametrize("partition", [0, 16, 32, 48, 80, 256, 1024, 4096])
def test_decode_tiny_partitions(uq, tiny_case, partition):
    wl, desc, codes, scales, ref = tiny_case
    log(f"decode tiny partition={partition}")
    out = run_decode(uq, wl, desc, codes, scales, torch.device("cuda:0"), partition=partition)
    check_attention(out, ref, f"tiny p={partition}")


def test_decode_tiny_dtypes(uq, tiny_case):
    wl, desc, codes, scales, ref = tiny_case
    dev = torch.device("cuda:0")
    out_bf = run_decode(uq, wl, desc, codes, scales, dev, out_dtype=torch.bfloat16)
    # a bf16 output adds one rounding of the result (relative 2^-9)
    assert np.all(np.abs(out_bf - ref) <= MAX_ABS + np.abs(ref) * 2.0 ** -8)
    q8 = uq.prepare_query(desc, wl.q.to(dev))
    out_fp8 = run_decode(uq, wl, desc, codes, scales, dev, q=q8, q_dtype=uq.UQ_FP8_E4M3)
    out_f32 = run_decode(uq, wl, desc, codes, scales, dev)
    assert np.array_equal(out_fp8, out_f32)
    qb = wl.q.bfloat16()
    pools, pt = oracle_cache(wl, [0], dev)
    ref_b = oracle.decode_attention(qb.float().numpy(), pools, pt, wl.context_lens, 1, 1 / math.sqrt(128), True)
    check_attention(run_decode(uq, wl, desc, codes, scales, dev, q=qb), ref_b, "tiny bf16 q")


@pytest.mark.parametrize("rotate_v", [True, False])
@pytest.mark.parametrize("partition", [0, 64])
def test_decode_ragged_gqa6(uq, rotate_v, partition):
    dev = torch.device("cuda:0")
    wl = workloads.custom(4, 12, 2, [1, 17, 1000, 0], seed=21, paging="random", rotate_v=rotate_v)
    log(f"decode ragged G=6 rotate_v={rotate_v} partition={partition}")
    desc, codes, scales = gpu_cache(uq, wl, dev)
    out = run_decode(uq, wl, desc, codes, scales, dev, partition=partition)
    pools, pt = oracle_cache(wl, list(range(wl.batch)), dev)
    ref = oracle.decode_attention(wl.q.numpy(), pools, pt, wl.context_lens, wl.num_kv_heads, 1 / math.sqrt(128),
                                  rotate_v)
    assert np.all(out[3] == 0)   # empty context
    check_attention(out, ref, f"ragged rv={rotate_v} p={partition}")


@pytest.mark.parametrize("hq,hkv", [(16, 1), (2, 2), (48, 3)])
def test_decode_group_sizes(uq, hq, hkv):
    dev = torch.device("cuda:0")
    wl = workloads.custom(2, hq, hkv, [300, 77], seed=5, paging="random")
    log(f"decode groups hq={hq} hkv={hkv}")
    desc, codes, scales = gpu_cache(uq, wl, dev)
    out = run_decode(uq, wl, desc, codes, scales, dev, partition=64)
    pools, pt = oracle_cache(wl, [0, 1], dev)
    ref = oracle.decode_attention(wl.q.numpy(), pools, pt, wl.context_lens, hkv, 1 / math.sqrt(128), True)
    check_attention(out, ref, f"groups {hq}/{hkv}")


def test_decode_long_partition_waves_reload_ids(uq):
    """Partitions of 16384 tokens: each of a block's waves walks more than
    32 page pairs, so it takes its later page ids from its LDS slot; a group
    of 16 fills every query row of the block.  One context held whole by one
    block, one split over two partitions, one ragged; against the oracle."""
    dev = torch.device("cuda:0")
    wl = workloads.custom(3, 16, 1, [16384, 20000, 9001], seed=41, paging="random")
    log("decode 16384-token partitions, G=16")
    desc, codes, scales = gpu_cache(uq, wl, dev)
    out = run_decode(uq, wl, desc, codes, scales, dev, partition=16384)
    pools, pt = oracle_cache(wl, [0, 1, 2], dev)
    ref = oracle.decode_attention(wl.q.numpy(), pools, pt, wl.context_lens, 1, 1 / math.sqrt(128), True)
    check_attention(out, ref, "16384-token partitions")


def test_decode_minimax_full_size_sampled(uq):
    """B=64, Hq=48, Hkv=8, lognormal contexts 8k..128k, a 16k-token prefix
    shared by every sequence (shorter contexts own a copy of their last
    page), the default partition: the shortest and the longest sequence
    against the oracle."""
    dev = torch.device("cuda:0")
    wl = workloads.minimax_like()
    log("decode minimax-like full size")
    desc, codes, scales = gpu_cache(uq, wl, dev, fill=None)
    out = run_decode(uq, wl, desc, codes, scales, dev)
    seqs = [int(np.argmin(wl.context_lens)), int(np.argmax(wl.context_lens))]
    pools, ptc = oracle_cache(wl, seqs, dev)
    ref = oracle.decode_attention(wl.q.numpy()[seqs], pools, ptc, wl.context_lens[seqs], wl.num_kv_heads,
                                  1 / math.sqrt(128), True)
    check_attention(out[seqs], ref, "minimax sampled")


def test_decode_high_concurrency_sampled(uq):
    """B=256, Hq=64, Hkv=8, every context 131072 (36.5 GB of FP4 KV),
    partitions of 4096 (the one-wave-per-partition grid, as the benchmark
    runs it): the first, last and two other sequences against the oracle."""
    dev = torch.device("cuda:0")
    wl = workloads.high_concurrency()
    log("decode high-concurrency full size")
    desc, codes, scales = gpu_cache(uq, wl, dev, fill=None)
    out = run_decode(uq, wl, desc, codes, scales, dev)
    del codes, scales
    torch.cuda.empty_cache()
    seqs = [0, 77, 201, 255]
    pools, ptc = oracle_cache(wl, seqs, dev)
    ref = oracle.decode_attention(wl.q.numpy()[seqs], pools, ptc, wl.context_lens[seqs], wl.num_kv_heads,
                                  1 / math.sqrt(128), True)
    check_attention(out[seqs], ref, "high-concurrency sampled")


def test_decode_qwen_full_size_sampled(uq):
    """B=32, Hq=64, Hkv=4, context 32768, random pages: the default launch
    configuration, checked on sampled sequences; deterministic across runs
    and across reuse of one workspace."""
    dev = torch.device("cuda:0")
    wl = workloads.qwen3_235b_like()
    log("decode qwen3-235b-like full size")
    desc, codes, scales = gpu_cache(uq, wl, dev, fill=None)
    out1 = run_decode(uq, wl, desc, codes, scales, dev)
    out2 = run_decode(uq, wl, desc, codes, scales, dev)
    assert np.array_equal(out1, out2)
    # the same workspace reused by many calls keeps giving the same answer
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    ws = uq.alloc_workspace(desc, wl.batch, wl.num_q_heads, wl.max_context)
    for _ in range(3):
        out3 = uq.decode_attention(desc, q, codes, scales, pt, ctx, wl.max_context, 1 / math.sqrt(128), workspace=ws)
    torch.cuda.synchronize()
    assert np.array_equal(out3.cpu().numpy(), out1)
    # the two launches called one by one give the same result
    part = uq.default_partition(desc, wl.batch, wl.num_q_heads, wl.max_context)
    out4 = torch.empty_like(q)
    uq.decode_partials(desc, q, codes, scales, pt, ctx, wl.max_context, 1 / math.sqrt(128), part, ws, out4)
    uq.decode_merge(desc, wl.batch, wl.num_q_heads, ctx, wl.max_context, part, ws, out4)
    torch.cuda.synchronize()
    assert np.array_equal(out4.cpu().numpy(), out1)
    seqs = [0, 19]
    pools, ptc = oracle_cache(wl, seqs, dev)
    ref = oracle.decode_attention(wl.q.numpy()[seqs], pools, ptc, wl.context_lens[seqs], wl.num_kv_heads,
                                  1 / math.sqrt(128), True)
    check_attention(out1[seqs], ref, "qwen sampled")
