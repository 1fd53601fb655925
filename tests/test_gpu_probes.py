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
