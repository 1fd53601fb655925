"""The measurement probes run on the GPU and read what they are asked to
read: the stream probe's block checksums fold every 32-bit word of the
buffer exactly once; the page-gather probe writes one checksum per wave of
the decode kernel's grid (0 for a wave with no pages)."""
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


@pytest.mark.parametrize("nbytes", [16, 4096 + 48, 64 << 20])
def test_stream_read_folds_every_word(uq, nbytes):
    dev = torch.device("cuda:0")
    g = torch.Generator(device=dev).manual_seed(nbytes)
    buf = torch.randint(0, 256, (nbytes,), dtype=torch.uint8, generator=g, device=dev)
    sink = uq.probe_stream_read(buf)
    torch.cuda.synchronize()
    words = buf.cpu().numpy().view(np.uint32)
    assert np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32)) == np.bitwise_xor.reduce(words)


def test_page_gather_writes_every_wave(uq):
    dev = torch.device("cuda:0")
    wl = workloads.custom(3, 16, 2, [2000, 0, 70], seed=41, paging="random")
    desc = uq.CacheDesc(num_kv_heads=2, num_pages=wl.num_pages)
    codes, scales = desc.alloc_pools(dev, fill=0)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
    part = 512
    nparts = -(-wl.max_context // part)
    sink = torch.full((4 * nparts * 2 * 3,), -1, dtype=torch.int32, device=dev)
    uq.probe_page_gather(desc, 16, codes, scales, torch.as_tensor(wl.page_table, device=dev),
                         torch.as_tensor(wl.context_lens, device=dev), wl.max_context, part, sink)
    torch.cuda.synchronize()
    s = sink.cpu().numpy().reshape(nparts, 3, 2, 4)   # [partition][sequence][kv head][wave]
    assert np.all(s != -1)
    assert np.all(s[:, 1] == 0)                        # the empty context
    assert np.all(s[1:, 2] == 0)                       # 70 tokens: one partition
    assert np.all(s[0, 2, :, 3] == 0)                  # ... of 5 pages: 3 page pairs for waves 0..2


def _fill(uq, wl, dev, head_dim=128):
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, head_dim=head_dim)
    codes, scales = desc.alloc_pools(dev, fill=0)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        if head_dim != 128:
            k, v = k[..., :head_dim].contiguous(), v[..., :head_dim].contiguous()
            if head_dim > 128:
                k = torch.cat([k, k.flip(-1)], -1)
                v = torch.cat([v, v.flip(-1)], -1)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
    return desc, codes, scales


@pytest.mark.parametrize("head_dim,hq", [(64, 16), (64, 48), (256, 16)])
def test_page_gather_head_sizes(uq, head_dim, hq):
    """The probe runs the head-size-64 and -256 grids (two kv heads per block
    at head size 64 and group size 8): waves without pages write 0, the
    others a checksum of the staged bytes, the same on a second run."""
    dev = torch.device("cuda:0")
    print(f"page-gather probe: head size {head_dim}, {hq} query heads", flush=True)
    wl = workloads.custom(3, hq, 4, [2000, 0, 70], seed=43, paging="random")
    desc, codes, scales = _fill(uq, wl, dev, head_dim)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    part = 512
    nparts = -(-wl.max_context // part)
    units = 2 if (head_dim == 64 and hq // 4 <= 8) else 4     # kv heads per block row: pairs at head size 64
    n = 4 * nparts * units * 3
    sink = torch.full((4 * nparts * 4 * 3,), -1, dtype=torch.int32, device=dev)
    uq.probe_page_gather(desc, hq, codes, scales, pt, ctx, wl.max_context, part, sink)
    again = uq.probe_page_gather(desc, hq, codes, scales, pt, ctx, wl.max_context, part, sink.clone())
    torch.cuda.synchronize()
    s = sink.cpu().numpy()
    assert np.array_equal(s, again.cpu().numpy())
    assert np.all(s[n:] == -1)                          # past the launch: untouched
    s = s[:n].reshape(nparts, 3, units, 4)              # [partition][sequence][kv unit][wave]
    assert np.all(s[:, 1] == 0)                         # the empty context
    assert np.all(s[1:, 2] == 0)                        # 70 tokens: one partition
    assert np.all(s[0, 2, :, 3] == 0)                   # ... of 5 pages: 3 page pairs for waves 0..2
    assert np.count_nonzero(s[:, 0]) == s[:, 0].size    # 2000 tokens: every wave of every partition staged pages


def test_page_gather_cascade(uq):
    """The cascade probe runs the cascade's grid: the row list (context rows
    with work, longest first, then the prefix rows, then rows without work),
    context blocks after each sequence's prefix part, prefix blocks of 16
    columns.  Every block of the launch writes its 4 words (0 for a wave
    without pages), nothing past it; the prefix rows sit right after the
    context rows with work; two runs give the same words up to the order of
    context rows of equal length."""
    dev = torch.device("cuda:0")
    print("page-gather probe: cascade", flush=True)
    wl = workloads.custom(6, 12, 2, [20, 96, 97, 150, 400, 0], seed=31, paging="random", shared_prefix_tokens=96)
    desc, codes, scales = _fill(uq, wl, dev)
    lens = wl.prefix_lens()
    prefix = uq.SharedPrefix(torch.as_tensor(wl.prefix_pages.astype(np.int32), device=dev),
                             torch.as_tensor(lens, device=dev), wl.shared_prefix_tokens, 32)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    P, B, H = 128, 6, 2
    nparts = -(-wl.max_context // P)
    # context rows that stay in the row list (as the cascade computes them)
    with_work = 0
    for b in range(B):
        c = int(wl.context_lens[b])
        pl = min(int(lens[b]), wl.shared_prefix_tokens, c - 1)
        pl = (pl & ~15) if pl > 0 else 0
        for part in range(nparts):
            s0 = part * P
            if s0 + P <= pl:
                continue
            if max(s0, pl) < c or (c <= 0 and part == 0):
                with_work += 1
    prefix_rows = -(-B * 6 // 16) * (96 // 32)              # per kv head: column chunks x prefix partitions
    blocks = H * (nparts * B + prefix_rows)
    sink = torch.full((4 * blocks + 64,), -1, dtype=torch.int32, device=dev)
    a = uq.probe_page_gather_cascade(desc, 12, codes, scales, pt, ctx, wl.max_context, prefix, P, sink=sink)
    a = a.cpu().numpy().copy()
    b2 = uq.probe_page_gather_cascade(desc, 12, codes, scales, pt, ctx, wl.max_context, prefix, P,
                                      sink=torch.full_like(sink, -1)).cpu().numpy()
    assert np.all(a[4 * blocks:] == -1) and np.all(a[:4 * blocks] != -1)
    assert np.array_equal(np.sort(a), np.sort(b2))
    rows = a[:4 * blocks].reshape(nparts * B + prefix_rows, H, 4)    # [row of the list][kv head][wave]
    pre = rows[with_work:with_work + prefix_rows]
    # a prefix partition of 32 tokens is one page pair: wave 0 stages it
    assert np.all(pre[:, :, 0] != 0) and np.all(pre[:, :, 1:] == 0)
    assert np.all(rows[with_work + prefix_rows:] == 0)             # rows without work
    assert np.count_nonzero(rows[:with_work]) > 0
