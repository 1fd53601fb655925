"""Seeded synthetic workloads with the shapes of the paper's decode layers.

This module only draws random numbers and builds index tables; it holds none
of the method's arithmetic, so both the HIP path and the CPU oracle can take
their inputs from it.

Recipe (stands in for the paper's MiniMax-M2.5 / Qwen3-235B attention layers
and agent-trace contexts, which are not available):
  * K, V ~ N(0, 1) in fp32, with 4 outlier channels per KV head for K and 4
    for V (drawn without replacement from the 128 channels) multiplied by 20;
  * q ~ N(0, 1) in fp32;
  * pages of 16 tokens; page tables are identity (tiny case) or a random
    permutation of the page pool; the MiniMax-like case shares its first
    16384 tokens (1024 pages) between all sequences and draws contexts from
    lognormal(ln 32768, 0.8) clipped to [8192, 131072]; a context shorter
    than the shared prefix shares its first tokens and owns a copy of its
    last page (copy on write).
Rows for the offline fit of the scale constant: uniform unit vectors
(normalised N(0, I) draws, the rotated-unit-vector model of the paper's
codebook analysis) and key rows of the recipe above.

Small index tables, outlier channels and queries come from a CPU
``torch.Generator``; the bulk K/V of every sequence comes from its own
generator on the target device, seeded from (workload seed, sequence), so any
sequence can be regenerated alone.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch

HEAD_DIM = 128
PAGE = 16
OUTLIERS = 4
OUTLIER_GAIN = 20.0


@dataclass
class DecodeWorkload:
    name: str
    batch: int
    num_q_heads: int
    num_kv_heads: int
    context_lens: np.ndarray          # int32 [B]
    page_table: np.ndarray            # int32 [B, max_pages_per_seq]
    num_pages: int
    seed: int
    shared_prefix_tokens: int = 0     # tokens 0..n-1 of every sequence live in shared pages
    private_tail: np.ndarray = field(default=None)   # bool [B]: last page copied out of the shared prefix
    prefix_pages: np.ndarray = field(default=None)   # int64 [shared pages]: the shared prefix's pages
    partition_tokens: int = 0         # 0 = library default
    rotate_v: bool = True
    k_outliers: np.ndarray = field(default=None)   # int64 [Hkv, 4]
    v_outliers: np.ndarray = field(default=None)
    q: torch.Tensor = field(default=None)          # fp32 [B, Hq, head_dim] on the CPU
    head_dim: int = HEAD_DIM

    @property
    def max_context(self) -> int:
        return int(self.context_lens.max()) if self.batch else 0

    @property
    def max_pages_per_seq(self) -> int:
        return int(self.page_table.shape[1])

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def total_tokens(self) -> int:
        return int(self.context_lens.astype(np.int64).sum())

    def kv_bytes_fp4(self) -> int:
        """Logical KV bytes one decode step reads: 17 B per 32 channels of K
        and of V per token and kv head (136 B at head size 128)."""
        return self.total_tokens() * self.num_kv_heads * 17 * self.head_dim // 16

    # -- bulk data ---------------------------------------------------------
    def segments(self):
        """(key, first token, last token + 1, row) of every stored run of
        tokens: the shared prefix once (key -1, row None: its own page list),
        each sequence's own tokens (key b, row b), and, for a sequence
        whose context ends inside the shared prefix, the prefix tokens of its
        last page again (key -1, row b): that page is a private copy, so a
        decode step can append to it without touching pages others read."""
        out = []
        if self.shared_prefix_tokens:
            out.append((-1, 0, self.shared_prefix_tokens, None))
        for b in range(self.batch):
            ctx = int(self.context_lens[b])
            lo = min(self.shared_prefix_tokens, ctx)
            if self.private_tail is not None and self.private_tail[b]:
                out.append((-1, ((ctx - 1) // PAGE) * PAGE, ctx, b))
            if ctx > lo:
                out.append((b, lo, ctx, b))
        return out

    def sequence_segments(self, b: int):
        """(key, first token, last token + 1) covering tokens 0..len-1 of
        sequence b once each, in order."""
        ctx = int(self.context_lens[b])
        lo = min(self.shared_prefix_tokens, ctx)
        out = [(-1, 0, lo)] if lo > 0 else []
        if ctx > lo:
            out.append((b, lo, ctx))
        return out

    def prefix_lens(self) -> np.ndarray:
        """int32 [B]: tokens of each sequence that are read from the shared
        prefix pages (whole pages, all before the sequence's last token)."""
        ctx = self.context_lens.astype(np.int64)
        full = np.minimum(self.shared_prefix_tokens, ctx)
        if self.private_tail is not None:
            full = np.where(self.private_tail, np.maximum(ctx - 1, 0) // PAGE * PAGE, full)
        return full.astype(np.int32)

    def slots(self, key: int, lo: int, hi: int, row=None) -> np.ndarray:
        """Physical slots of tokens lo..hi-1 through page-table row `row`
        (None: the shared prefix's page list)."""
        pos = np.arange(lo, hi, dtype=np.int64)
        if row is None and key >= 0:
            row = key
        pages = self.prefix_pages[pos // PAGE] if row is None else self.page_table[row, pos // PAGE].astype(np.int64)
        return pages * PAGE + pos % PAGE

    def kv(self, key: int, lo: int, hi: int, device="cpu", dtype=torch.float32):
        """K, V [hi-lo, Hkv, head_dim] of one segment, regenerated from its own
        seed.  A sequence's stream (key >= 0) starts at the segment; the
        shared prefix (key -1) is always drawn whole and then sliced, so any
        part of it can be regenerated (a generator's leading values depend
        on the size of the draw)."""
        g = torch.Generator(device=device)
        g.manual_seed(self.seed * 1_000_003 + (key + 1))
        if key < 0:
            assert 0 <= lo <= hi <= self.shared_prefix_tokens
            n, skip = self.shared_prefix_tokens, lo
        else:
            n, skip = hi - lo, 0
        k = torch.randn((n, self.num_kv_heads, self.head_dim), generator=g, device=device, dtype=torch.float32)
        v = torch.randn((n, self.num_kv_heads, self.head_dim), generator=g, device=device, dtype=torch.float32)
        k, v = k[skip:skip + hi - lo], v[skip:skip + hi - lo]
        for h in range(self.num_kv_heads):
            k[:, h, torch.as_tensor(self.k_outliers[h], device=device)] *= OUTLIER_GAIN
            v[:, h, torch.as_tensor(self.v_outliers[h], device=device)] *= OUTLIER_GAIN
        return k.to(dtype), v.to(dtype)


def _meta(gen: torch.Generator, wl: DecodeWorkload):
    d = wl.head_dim
    wl.k_outliers = np.stack([torch.randperm(d, generator=gen)[:OUTLIERS].numpy() for _ in range(wl.num_kv_heads)])
    wl.v_outliers = np.stack([torch.randperm(d, generator=gen)[:OUTLIERS].numpy() for _ in range(wl.num_kv_heads)])
    wl.q = torch.randn((wl.batch, wl.num_q_heads, d), generator=gen, dtype=torch.float32)
    return wl


def custom(batch, num_q_heads, num_kv_heads, context_lens, seed=0, paging="random", spare_pages=3,
           shared_prefix_tokens=0, partition_tokens=0, rotate_v=True, name="custom", head_dim=HEAD_DIM) -> DecodeWorkload:
    """A decode workload of any shape (head_dim 64, 128 or 256): paging
    'identity' or 'random'."""
    ctx = np.asarray(context_lens, dtype=np.int32).reshape(batch)
    gen = torch.Generator().manual_seed(seed)
    pages_per = [(int(c) + PAGE - 1) // PAGE for c in ctx]
    maxp = max(1, max(pages_per))
    shared = shared_prefix_tokens // PAGE
    assert shared_prefix_tokens % PAGE == 0
    own = [max(0, p - shared) for p in pages_per]
    # a context that ends inside the shared prefix gets a private copy of its
    # last page (copy on write), so that appends never touch shared pages
    tail = np.array([0 < pages_per[b] <= shared for b in range(batch)], dtype=bool)
    num_pages = shared + sum(own) + int(tail.sum()) + spare_pages
    if paging == "identity":
        perm = np.arange(num_pages, dtype=np.int64)
    else:
        perm = torch.randperm(num_pages, generator=gen).numpy()
    pt = np.full((batch, maxp), -1, dtype=np.int32)
    cur = shared
    for b in range(batch):
        n_sh = min(shared, pages_per[b])
        pt[b, :n_sh] = perm[:n_sh]
        pt[b, n_sh:pages_per[b]] = perm[cur:cur + own[b]]
        cur += own[b]
        if tail[b]:
            pt[b, pages_per[b] - 1] = perm[cur]
            cur += 1
    pt[pt < 0] = 0   # unused entries point at a valid page; they are never read
    wl = DecodeWorkload(name, batch, num_q_heads, num_kv_heads, ctx, pt, num_pages, seed,
                        shared_prefix_tokens=shared_prefix_tokens, partition_tokens=partition_tokens,
                        rotate_v=rotate_v, private_tail=tail if tail.any() else None,
                        prefix_pages=np.asarray(perm[:shared], dtype=np.int64), head_dim=head_dim)
    return _meta(gen, wl)


def tiny() -> DecodeWorkload:
    """1 sequence, 1 KV head, 8 query heads, context 4096, identity pages, seed 0."""
    return custom(1, 8, 1, [4096], seed=0, paging="identity", spare_pages=0, name="tiny-gqa8-ctx4096")


def qwen3_235b_like() -> DecodeWorkload:
    """64 query heads, 4 KV heads, batch 32, every context 32768, random pages."""
    return custom(32, 64, 4, [32768] * 32, seed=1, paging="random", spare_pages=0, name="qwen3-235b-like-b32-ctx32k")


def minimax_like() -> DecodeWorkload:
    """48 query heads, 8 KV heads, batch 64, lognormal contexts 8k..128k, 16k shared prefix."""
    gen = torch.Generator().manual_seed(2)
    z = torch.randn(64, generator=gen, dtype=torch.float64).numpy()
    ctx = np.clip(np.rint(np.exp(math.log(32768) + 0.8 * z)), 8192, 131072).astype(np.int32)
    return custom(64, 48, 8, ctx, seed=2, paging="random", spare_pages=0, shared_prefix_tokens=16384,
                  name="minimax-like-b64-lognormal-shared16k")


def high_concurrency() -> DecodeWorkload:
    """64 query heads, 8 KV heads, batch 256, every context 131072, partitions of 4096."""
    return custom(256, 64, 8, [131072] * 256, seed=4, paging="random", spare_pages=0, partition_tokens=4096,
                  name="high-concurrency-b256-ctx128k")


@dataclass
class WriteWorkload:
    """Quantize-on-write: a 65536-token prefill into random pages, then a
    1-token append for each of 256 sequences through a page table."""
    num_kv_heads: int = 8
    prefill_tokens: int = 65536
    append_seqs: int = 256
    num_pages: int = 8192
    max_pages_per_seq: int = 512
    seed: int = 3

    def build(self, device="cpu", dtype=torch.bfloat16):
        gen = torch.Generator().manual_seed(self.seed)
        perm = torch.randperm(self.num_pages, generator=gen).numpy()
        pre_pages = self.prefill_tokens // PAGE
        pos = np.arange(self.prefill_tokens, dtype=np.int64)
        prefill_slots = perm[pos // PAGE].astype(np.int64) * PAGE + pos % PAGE
        ctx = torch.randint(1, 8192, (self.append_seqs,), generator=gen).numpy().astype(np.int64)
        pt = np.zeros((self.append_seqs, self.max_pages_per_seq), dtype=np.int32)
        for s in range(self.append_seqs):
            pt[s, ctx[s] // PAGE] = perm[pre_pages + s]
        append_slots = np.arange(self.append_seqs, dtype=np.int64) * self.max_pages_per_seq * PAGE + ctx
        ko = np.stack([torch.randperm(HEAD_DIM, generator=gen)[:OUTLIERS].numpy() for _ in range(self.num_kv_heads)])
        vo = np.stack([torch.randperm(HEAD_DIM, generator=gen)[:OUTLIERS].numpy() for _ in range(self.num_kv_heads)])
        g = torch.Generator(device=device).manual_seed(self.seed * 1_000_003)

        def draw(n):
            k = torch.randn((n, self.num_kv_heads, HEAD_DIM), generator=g, device=device)
            v = torch.randn((n, self.num_kv_heads, HEAD_DIM), generator=g, device=device)
            for h in range(self.num_kv_heads):
                k[:, h, torch.as_tensor(ko[h], device=device)] *= OUTLIER_GAIN
                v[:, h, torch.as_tensor(vo[h], device=device)] *= OUTLIER_GAIN
            return k.to(dtype), v.to(dtype)

        kp, vp = draw(self.prefill_tokens)
        ka, va = draw(self.append_seqs)
        return dict(prefill=(kp, vp, prefill_slots), append=(ka, va, append_slots, pt, ctx))


def unit_vectors(n: int, d: int, seed: int = 0) -> np.ndarray:
    """n uniform unit vectors in R^d (fp32 [n, d]): N(0, I) rows divided by
    their norms, from numpy's PCG64 seeded with ``seed``."""
    g = np.random.default_rng(seed).standard_normal((n, d))
    return (g / np.linalg.norm(g, axis=1, keepdims=True)).astype(np.float32)


def key_rows(n: int, seed: int = 0) -> np.ndarray:
    """n key rows of 128 channels (fp32 [n, 128]) with the cache recipe:
    N(0, 1) with 4 outlier channels (the same for every row) times 20."""
    rng = np.random.default_rng(seed)
    k = rng.standard_normal((n, HEAD_DIM))
    k[:, rng.permutation(HEAD_DIM)[:OUTLIERS]] *= OUTLIER_GAIN
    return k.astype(np.float32)


def gpt_oss_like(head_dim: int = 64) -> DecodeWorkload:
    """A head-size-64 attention layer shaped like GPT-OSS-20B's (the model of
    the paper's per-block ablation): 64 query heads, 8 KV heads, batch 32,
    every context 32768, random pages; seed 5.  head_dim 256 gives the same
    shape at head size 256 (seed 6)."""
    return custom(32, 64, 8, [32768] * 32, seed=5 if head_dim == 64 else 6, paging="random", spare_pages=0,
                  name=f"gpt-oss-like-hd{head_dim}-b32-ctx32k", head_dim=head_dim)
