"""Scores far outside the usual range: keys scaled by 2^e (f32 rows, so the
scale bytes reach 127 + e and the raw scores about 2^(e+3)) at head sizes
64 (one and two heads per block), 128 and 256, against the oracle.  The
running softmax max is kept above the exact scaled scores, so no exponent
overflows; at these magnitudes the softmax is close to one-hot, which the
fp64 oracle reproduces within the usual tolerances."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


@pytest.mark.parametrize("d,hq,hkv", [(64, 8, 2), (64, 3, 3), (128, 16, 2), (256, 8, 1)])
@pytest.mark.parametrize("e", [0, 16, 34, 60])
def test_scaled_keys(uq, d, hq, hkv, e):
    print(f"range d={d} hq={hq} hkv={hkv} keys x 2^{e}", flush=True)
    dev = torch.device("cuda:0")
    wl = workloads.custom(3, hq, hkv, [700, 37, 300], seed=71, paging="random", head_dim=d)
    desc = uq.CacheDesc(num_kv_heads=hkv, num_pages=wl.num_pages, rotate_v=True, head_dim=d)
    codes, scales = desc.alloc_pools(dev, fill=0)
    pools = oracle.alloc_pools(wl.num_pages, hkv, fill=0, head_dim=d)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        k = k * 2.0 ** e
        slots = wl.slots(key, lo, hi, row)
        uq.quantize_kv(desc, k, v, torch.as_tensor(slots, device=dev), codes, scales)
        oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), slots, wl.num_pages, rotate_v=True, pools=pools)
    torch.cuda.synchronize()
    assert np.array_equal(codes.cpu().numpy(), pools[0])
    assert np.array_equal(scales.cpu().numpy(), pools[1])
    for partition in (0, 64):
        out = uq.decode_attention(desc, wl.q.to(dev), codes, scales, torch.as_tensor(wl.page_table, device=dev),
                                  torch.as_tensor(wl.context_lens, device=dev), wl.max_context, 1 / math.sqrt(d),
                                  partition)
        torch.cuda.synchronize()
        got = out.cpu().numpy().astype(np.float64)
        ref = oracle.decode_attention(wl.q.numpy(), pools, wl.page_table, wl.context_lens, hkv, 1 / math.sqrt(d),
                                      True)
        assert np.all(np.isfinite(got)), f"non-finite output, partition {partition}"
        err = np.abs(got - ref).max()
        rel = np.linalg.norm(got - ref) / np.linalg.norm(ref)
        print(f"  partition {partition}: max-abs {err:.2e} rel-L2 {rel:.2e}", flush=True)
        assert err <= 2e-3 and rel <= 1e-3
