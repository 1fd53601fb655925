"""Host logic of bench.py: the algorithmic byte count it divides by, the
single-GPU contract, and the profile lookup."""
import os
import subprocess
import sys

import numpy as np

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from paper_2606_20474_amd import workloads  # noqa: E402


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_token_heads_plain_and_cascade():
    wl = workloads.qwen3_235b_like()
    assert bench.alg_token_heads(wl, False) == 32 * 32768 * 4
    mm = workloads.minimax_like()
    # brute force: the distinct (page, kv head) token slots a cascade launch reads
    shared = set(int(p) for p in mm.prefix_pages)
    own = 0
    for b in range(mm.batch):
        n = int(mm.context_lens[b])
        pl = int(mm.prefix_lens()[b])
        own += n - pl
        assert all(int(p) in shared for p in mm.page_table[b, :pl // 16])
    assert bench.alg_token_heads(mm, True) == (own + mm.shared_prefix_tokens) * mm.num_kv_heads
    assert bench.alg_token_heads(mm, False) == int(mm.context_lens.astype(np.int64).sum()) * mm.num_kv_heads


def test_bytes_per_token_head_match_the_pools():
    """136 B per (token, kv head) is what the pools hold per token (codes and
    scale bytes), and the comparison caches' 256 / 512 / 148 B likewise."""
    from paper_2606_20474_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    from paper_2606_20474_amd import uq
    d = uq.CacheDesc(num_kv_heads=3, num_pages=7)
    assert (d.codes_bytes() + d.scales_bytes()) == 7 * 3 * 16 * bench.KV_BYTES_PER_TOKEN_HEAD
    for fmt in ("fp8", "bf16", "tq4"):
        r = uq.RefCacheDesc(3, 7, fmt)
        assert r.cache_bytes() == 7 * 3 * 16 * bench.REF_BYTES_PER_TOKEN_HEAD[fmt], fmt


def test_profile_lookup_without_a_profile_is_none():
    assert bench.profiled_traffic("no-such-workload") is None
