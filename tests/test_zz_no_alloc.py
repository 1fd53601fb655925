"""uq_decode_attention_noalloc (through the C ABI) against
uq_decode_attention: the same kernels and launch configuration with the
partials in the library's own device array instead of a workspace, so the
outputs must be identical bit for bit.  Two calls in a row, the second on a
smaller input, so that the array holds the first call's partials when the
second one runs."""
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


def log(msg):
    print(msg, flush=True)


def cache(uq, wl, dev, head_dim=128):
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v,
                        head_dim=head_dim)
    codes, scales = desc.alloc_pools(dev, fill=0)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
    return desc, codes, scales


def both(uq, wl, desc, codes, scales, dev, part):
    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    scale = 1 / math.sqrt(desc.head_dim)
    ref = uq.decode_attention(desc, q, codes, scales, pt, ctx, wl.max_context, scale, part)
    out = torch.full_like(ref, float("nan"))
    uq.decode_attention_noalloc(desc, q, codes, scales, pt, ctx, wl.max_context, out, scale, part)
    torch.cuda.synchronize()
    return out.cpu().numpy(), ref.cpu().numpy()


@pytest.mark.parametrize("part", [0, 256])
def test_noalloc_equals_workspace_call_twice(uq, part):
    dev = torch.device("cuda:0")
    big = workloads.custom(6, 32, 4, [9000, 1, 4097, 0, 2500, 17], seed=31, paging="random")
    small = workloads.custom(2, 16, 2, [700, 33], seed=32, paging="random")
    for name, wl in (("first, larger", big), ("second, smaller", small)):
        log(f"noalloc vs workspace: {name} B={wl.batch} Hq={wl.num_q_heads} Hkv={wl.num_kv_heads} part={part}")
        desc, codes, scales = cache(uq, wl, dev)
        out, ref = both(uq, wl, desc, codes, scales, dev, part)
        assert np.all(np.isfinite(out))
        assert np.array_equal(out, ref), (name, np.abs(out - ref).max())


def test_noalloc_head_size_64_and_oversize(uq):
    dev = torch.device("cuda:0")
    wl = workloads.custom(3, 16, 2, [3000, 640, 5], seed=33, paging="random", head_dim=64)
    log("noalloc vs workspace: head size 64")
    desc, codes, scales = cache(uq, wl, dev, head_dim=64)
    out, ref = both(uq, wl, desc, codes, scales, dev, 64)
    assert np.array_equal(out, ref)
    # more partials than the array holds: refused before anything runs
    big_q = torch.zeros((400, 16, 64), device=dev)
    big_pt = torch.zeros((400, 8192), dtype=torch.int32, device=dev)
    big_ctx = torch.zeros(400, dtype=torch.int32, device=dev)
    big_out = torch.zeros((400, 16, 64), device=dev)
    assert uq.workspace_bytes(desc, 400, 16, 131072, 1024) > uq.NOALLOC_SCRATCH_BYTES
    with pytest.raises(uq.UQError) as e:
        uq.decode_attention_noalloc(desc, big_q, codes, scales, big_pt, big_ctx, 131072, big_out, 0.125, 1024)
    assert e.value.status == uq.UQ_ERR_WORKSPACE_TOO_SMALL
    torch.cuda.synchronize()
    assert np.all(big_out.cpu().numpy() == 0)   # nothing was launched


def test_noalloc_wave_grid_then_block_grid(uq):
    """The one-wave-per-partition grid (40 sequences x 4 kv heads x 16 blocks
    of eight 16-token partitions, group 2: 21 MB of partials), then a call
    on the block grid."""
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(34)
    ctx = [0, 1, 31, 32, 33, 2048, 2047, 100] + [int(c) for c in rng.integers(1, 2049, 32)]
    wave = workloads.custom(40, 8, 4, ctx, seed=34, paging="random")
    small = workloads.custom(3, 12, 2, [300, 0, 77], seed=35, paging="random")
    for name, wl, part in (("wave grid", wave, 16), ("block grid", small, 64)):
        log(f"noalloc vs workspace: {name} B={wl.batch} Hq={wl.num_q_heads} Hkv={wl.num_kv_heads} part={part}")
        desc, codes, scales = cache(uq, wl, dev)
        out, ref = both(uq, wl, desc, codes, scales, dev, part)
        assert np.all(np.isfinite(out))
        assert np.array_equal(out, ref), (name, np.abs(out - ref).max())
