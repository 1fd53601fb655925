"""The PV-on-the-block-scaled-instruction prototype (uq_decode_attention_scaled_pv)
against the oracle, through the C ABI: the same bar as the default path
(max-abs 2e-3, relative L2 1e-3, Algorithm 1, Decode), on the tiny workload
at several partitions (in place, split, partial 128-token super-iterations),
ragged contexts with an empty one, both V modes, several group shapes and
query dtypes, and sampled sequences of the full Qwen3-235B-like layer."""
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


def check(got, ref, what):
    got = np.asarray(got, np.float64)
    err = np.abs(got - ref)
    rel = np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-30)
    log(f"{what}: max-abs {err.max():.3e} rel-L2 {rel:.3e}")
    assert np.all(np.isfinite(got)), what
    assert err.max() <= MAX_ABS, (what, err.max())
    assert rel <= REL_L2, (what, rel)


def caches(uq, wl, dev, seqs):
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v)
    codes, scales = desc.alloc_pools(dev, fill=0xA5)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.quantize_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), codes, scales)
    maxp = wl.max_pages_per_seq
    pt = np.arange(len(seqs) * maxp, dtype=np.int32).reshape(len(seqs), maxp)
    pools = oracle.alloc_pools(len(seqs) * maxp, wl.num_kv_heads)
    for i, b in enumerate(seqs):
        for key, lo, hi in wl.sequence_segments(b):
            k, v = wl.kv(key, lo, hi, device=dev)
            pos = np.arange(lo, hi, dtype=np.int64)
            oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), pt[i, pos // 16].astype(np.int64) * 16 + pos % 16,
                               len(seqs) * maxp, rotate_v=wl.rotate_v, pools=pools)
    torch.cuda.synchronize()
    return desc, codes, scales, pools, pt


def run(uq, wl, desc, codes, scales, dev, part, q=None):
    q = wl.q if q is None else q
    out = uq.decode_attention_scaled_pv(desc, q.to(dev), codes, scales, torch.as_tensor(wl.page_table, device=dev),
                                        torch.as_tensor(wl.context_lens, device=dev), wl.max_context,
                                        1 / math.sqrt(128), part)
    torch.cuda.synchronize()
    return out.float().cpu().numpy()


@pytest.mark.parametrize("part", [0, 32, 96, 256, 1024])
def test_tiny(uq, part):
    dev = torch.device("cuda:0")
    wl = workloads.tiny()
    log(f"scaled PV, tiny, partition {part}")
    desc, codes, scales, pools, pt = caches(uq, wl, dev, [0])
    ref = oracle.decode_attention(wl.q.numpy(), pools, pt, wl.context_lens, 1, 1 / math.sqrt(128), True)
    check(run(uq, wl, desc, codes, scales, dev, part), ref, f"tiny p={part}")


@pytest.mark.parametrize("rotate_v", [True, False])
@pytest.mark.parametrize("qdt", [torch.float32, torch.bfloat16])
def test_ragged_gqa6(uq, rotate_v, qdt):
    dev = torch.device("cuda:0")
    wl = workloads.custom(4, 12, 2, [1, 17, 1000, 0], seed=21, paging="random", rotate_v=rotate_v)
    log(f"scaled PV, ragged G=6 rotate_v={rotate_v} q {qdt}")
    desc, codes, scales, pools, pt = caches(uq, wl, dev, list(range(4)))
    q = wl.q.to(qdt)
    ref = oracle.decode_attention(q.float().numpy(), pools, pt, wl.context_lens, 2, 1 / math.sqrt(128), rotate_v)
    for part in (0, 64):
        out = run(uq, wl, desc, codes, scales, dev, part, q=q)
        assert np.all(out[3] == 0)
        check(out, ref, f"ragged rv={rotate_v} p={part}")


@pytest.mark.parametrize("hq,hkv", [(16, 1), (2, 2), (48, 3)])
def test_group_sizes(uq, hq, hkv):
    dev = torch.device("cuda:0")
    wl = workloads.custom(2, hq, hkv, [700, 77], seed=5, paging="random")
    log(f"scaled PV, groups {hq}/{hkv}")
    desc, codes, scales, pools, pt = caches(uq, wl, dev, [0, 1])
    ref = oracle.decode_attention(wl.q.numpy(), pools, pt, wl.context_lens, hkv, 1 / math.sqrt(128), True)
    check(run(uq, wl, desc, codes, scales, dev, 64), ref, f"groups {hq}/{hkv}")


def test_qwen_full_size_sampled(uq):
    dev = torch.device("cuda:0")
    wl = workloads.qwen3_235b_like()
    log("scaled PV, qwen3-235b-like full size")
    seqs = [0, 19]
    desc, codes, scales, pools, pt = caches(uq, wl, dev, seqs)
    out = run(uq, wl, desc, codes, scales, dev, 0)
    base = uq.decode_attention(desc, wl.q.to(dev), codes, scales, torch.as_tensor(wl.page_table, device=dev),
                               torch.as_tensor(wl.context_lens, device=dev), wl.max_context, 1 / math.sqrt(128))
    torch.cuda.synchronize()
    ref = oracle.decode_attention(wl.q.numpy()[seqs], pools, pt, wl.context_lens[seqs], wl.num_kv_heads,
                                  1 / math.sqrt(128), True)
    check(out[seqs], ref, "qwen sampled")
    check(out, base.cpu().numpy().astype(np.float64), "qwen, against the BF16 PV path")
