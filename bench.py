"""Decode-step benchmark of the FP4 KV path on one MI355X.

One step is the whole hot path for one decode token per sequence, the two
launches of uq_decode_step:
  1. uq_decode_step_partials writes the step's new K/V token of every
     sequence into the FP4 cache at the last position of its context
     (Algorithm 1, "Write"; done by the block that reads that page) and runs
     the partition kernel of decode attention over the full contexts
     (Algorithm 1, "Decode");
  2. uq_decode_merge merges the partitions.
For a workload whose sequences share a prefix (minimax-like), the step is
the same pair of launches of uq_decode_cascade: the prefix pages are read
once per kv head for 16 (sequence, query head) columns at a time.
Inputs are resident in HBM before the timed region.  The default workload is
the Qwen3-235B-like layer: 64 query heads, 4 KV heads, head_dim 128, batch
32, every context 32768, random page table.  ``value`` is KV tokens/s =
sum of contexts / step time.

The JSON line also carries the roofline of the dominant kernel (the decode
kernel: algorithmic KV bytes per launch / its mean launch time from HIP
events on its stream), the CPU oracle timed on a sample of the same
workload, and the same step over the comparison caches (FP8 E4M3 with
per-tensor scales, 256 B per token and kv head; BF16, 512 B; the Ultra-TQ
codebook cache, 148 B), built by the same library with the same decode
kernel and timed the same way.

The gpt-oss-like workloads run the FP4 path at head sizes 64 and 256 (64
query heads, 8 KV heads, batch 32, context 32768): there the step writes the
new tokens with uq_quantize_kv, then runs uq_decode_partials and
uq_decode_merge (the fused step and the comparison caches are head-size-128
calls).
"""
import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
KV_BYTES_PER_TOKEN_HEAD = 136   # K and V: 2 x (64 B codes + 4 B scales)
REF_BYTES_PER_TOKEN_HEAD = {"fp8": 256, "bf16": 512, "tq4": 148}
REF_SCALE = 0.3                 # per-tensor FP8 scale of the comparison cache (|x| up to 134 representable)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    # after an idle spell the first ~100 launches (about 12 ms of steps) run
    # up to 5 % slower while the GPU leaves its idle state
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default="qwen3-235b-like",
                    choices=["qwen3-235b-like", "high-concurrency", "minimax-like", "tiny", "gpt-oss-like-hd64",
                             "gpt-oss-like-hd256"])
    ap.add_argument("--partition", type=int, default=-1, help="partition tokens (-1: workload default)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-seqs", type=int, default=8)
    ap.add_argument("--comparators", default="fp8,bf16,tq4",
                    help="comma list of comparison caches to time as well (fp8, bf16, tq4) or 'none'")
    ap.add_argument("--no-cascade", action="store_true",
                    help="workloads with a shared prefix: read it per sequence instead of once per kv head")
    ap.add_argument("--no-write-path", action="store_true",
                    help="skip the quantize-on-write measurement (65536-token bf16 prefill + 256 appends)")
    ap.add_argument("--no-flush", action="store_true",
                    help="time the FP4 decode kernel back to back only (no 1 GiB write between launches)")
    ap.add_argument("--no-probes", action="store_true", help="skip the achievable-bandwidth probes")
    ap.add_argument("--no-scaled-pv", action="store_true",
                    help="skip the A/B of PV on the block-scaled instruction (head size 128 only)")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one device-to-device copy of this many MiB before the timed steps; its "
                         "FETCH_SIZE/WRITE_SIZE counters calibrate the HBM-traffic counters")
    return ap.parse_args()


def progress(msg):
    """One line on stderr per finished stage (stdout carries only the JSON line)."""
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def make_workload(name):
    from paper_2606_20474_amd import workloads
    return {"qwen3-235b-like": workloads.qwen3_235b_like, "high-concurrency": workloads.high_concurrency,
            "minimax-like": workloads.minimax_like, "tiny": workloads.tiny,
            "gpt-oss-like-hd64": lambda: workloads.gpt_oss_like(64),
            "gpt-oss-like-hd256": lambda: workloads.gpt_oss_like(256)}[name]()


def kernel_source_hash():
    """sha256 of the decode kernel's sources without comments and layout
    (a change to a comment does not change the kernel); a profile taken on
    other sources is stale."""
    import hashlib
    import re
    h = hashlib.sha256()
    for name in ("uq_decode.hip", "uq_device.hpp"):
        with open(os.path.join(ROOT, "paper_2606_20474_amd", "csrc", name)) as f:
            text = f.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def profiled_traffic(workload_name, fmt="fp4"):
    """HBM bytes per decode-kernel launch (fmt: fp4, fp8 or bf16 cache) from
    the committed counter profile of this workload (FETCH_SIZE and
    WRITE_SIZE, calibrated against a copy of known size), or None when there
    is none for the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"decode_kernel_{workload_name}.md")
    if not os.path.exists(path):
        return None
    field = "traffic_bytes_per_launch" + ("" if fmt == "fp4" else f"_{fmt}")
    fields = {}
    with open(path) as f:
        for line in f:
            if ":" in line and (line.startswith("traffic_bytes_per_launch") or line.startswith("source_sha256:")):
                k, v = line.split(":", 1)
                fields[k.strip()] = v.strip()
    if fields.get("source_sha256") != kernel_source_hash():
        return None
    try:
        return float(fields[field])
    except (KeyError, ValueError):
        return None


def fill_cache(uq, wl, desc, codes, scales, dev):
    """Quantise every stored segment of the workload into the pools (setup, untimed)."""
    import torch
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        slots = torch.as_tensor(wl.slots(key, lo, hi, row), device=dev)
        uq.quantize_kv(desc, k, v, slots, codes, scales)
        del k, v
    torch.cuda.synchronize()


def alg_token_heads(wl, cascade):
    """(token, kv head) pairs one decode launch must read: every context
    whole, or with the cascade the shared prefix once per kv head plus each
    sequence's tokens after it."""
    if not cascade:
        return wl.total_tokens() * wl.num_kv_heads
    own = int((wl.context_lens.astype(np.int64) - wl.prefix_lens().astype(np.int64)).sum())
    return (own + wl.shared_prefix_tokens) * wl.num_kv_heads


FLUSH_BYTES = 1 << 30   # written and read between flushed steps: 4x the 256 MB last-level cache


def timed(step, steps, warmup, stream, flush=None):
    """Run `warmup` untimed steps, then `steps` timed ones twice; returns (ms
    per step, mean ms between the event pair each step hands to
    uq.time_next_launch, which brackets the timed kernel itself: the decode
    partition kernel, a probe or the quantize-on-write kernel, start to end,
    as rocprofv3 reports it).

    The step time comes from the first pass, whose launches carry no kernel
    events (a launch that records its own start and end events costs the
    step about 4 us); the kernel time from the second, the same steps with
    the events.  Without `flush` the steps run back to back and the step
    time is the whole timed region over `steps`.  With `flush` (a callable
    that writes FLUSH_BYTES of device memory), every timed step is preceded
    by that write and read, outside its events, so that no step finds the
    previous one's bytes in L2 or the last-level cache; the step time is then
    the mean over steps of an event pair recorded on the stream around the
    step's launches."""
    import gc
    import torch
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    around = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in evs + around:   # create the HIP events
        a.record(stream)
        b.record(stream)
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    # no Python garbage collection from the warmup to the end: a collection
    # pause on the host leaves the GPU idle, and after an idle spell its
    # first launches run slower (the warmup covers the start of the run)
    gc.collect()
    gc.disable()

    def one_pass(kernel_events):
        t_start.record(stream)
        for i in range(steps):
            if flush is not None:
                flush()
                around[i][0].record(stream)
            if kernel_events:
                step(*evs[i])
            else:
                step()
            if flush is not None:
                around[i][1].record(stream)
        t_end.record(stream)
        torch.cuda.synchronize()
        if flush is None:
            return t_start.elapsed_time(t_end) / steps
        return float(np.mean([a.elapsed_time(b) for a, b in around]))

    try:
        for _ in range(warmup):
            if flush is not None:
                flush()
            step()
        torch.cuda.synchronize()
        step_ms = one_pass(False)
        one_pass(True)
    finally:
        gc.enable()
    kernel_ms = float(np.mean([a.elapsed_time(b) for a, b in evs]))
    return step_ms, kernel_ms


def make_flush(dev):
    """1 GiB written, then read back (uq_probe_stream_read): the write evicts
    the workload's lines from L2 and the last-level cache, the read evicts
    the write's dirty lines in turn, so that their write-back to HBM happens
    here and not inside the next timed kernel (a write alone left up to
    256 MB of dirty lines behind and added ~60 us of write-back traffic to
    the next launch)."""
    import torch
    from paper_2606_20474_amd import uq
    buf = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)
    sink = torch.empty(uq.PROBE_STREAM_BLOCKS, dtype=torch.int32, device=dev)
    state = {"i": 0}

    def flush():
        state["i"] += 1
        buf.fill_(state["i"] & 0xFF)
        uq.probe_stream_read(buf, sink)
    return flush


def comparator(uq, fmt, wl, part, q, pt, ctx, k_new, v_new, args, dev, stream, flush, prefix=None):
    """The same step (uq_ref_decode_step: the new token of every sequence
    written by the partition launch, then the merge) over a comparison cache
    holding the same K/V: plain FP8 or BF16, or the Ultra-TQ codebook cache
    (148 B per token and kv head: 64 B of K indices, a 4 B norm, 64 B of V
    codes and 4 x 4 B of (scale, zero))."""
    import torch
    desc = uq.RefCacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, fmt=fmt, k_scale=REF_SCALE,
                           v_scale=REF_SCALE)
    cache = desc.alloc_cache(dev)
    for key, lo, hi, row in wl.segments():
        k, v = wl.kv(key, lo, hi, device=dev)
        uq.ref_write_kv(desc, k, v, torch.as_tensor(wl.slots(key, lo, hi, row), device=dev), cache)
        del k, v
    if prefix is None:
        ws = uq.ref_alloc_workspace(desc, wl.batch, wl.num_q_heads, wl.max_context, part, dev)
    else:
        ws = torch.empty(uq.cascade_workspace_bytes(wl.num_kv_heads, wl.batch, wl.num_q_heads, wl.max_context, prefix,
                                                    part), dtype=torch.uint8, device=dev)
    out = torch.empty((wl.batch, wl.num_q_heads, 128), dtype=torch.float32, device=dev)
    scale = 1 / math.sqrt(128)

    def step(ev_a=None, ev_b=None):
        if ev_a is not None:
            uq.time_next_launch(ev_a, ev_b)
        if prefix is None:
            uq.ref_decode_step(desc, q, k_new, v_new, cache, pt, ctx, wl.max_context, scale, part, ws, out,
                               partials_only=True)
        else:
            uq.ref_decode_cascade(desc, q, cache, pt, ctx, wl.max_context, prefix, scale, part, ws, out,
                                  k_new=k_new, v_new=v_new, partials_only=True)
        if prefix is None:
            uq.ref_decode_merge(desc, wl.batch, wl.num_q_heads, ctx, wl.max_context, part, ws, out)
        else:
            uq.ref_decode_cascade_merge(desc, wl.batch, wl.num_q_heads, ctx, wl.max_context, prefix, part, ws, out)

    ms_step, dec_ms = timed(step, args.steps, args.warmup, stream)
    f_step, f_dec = timed(step, args.steps, args.warmup, stream, flush=flush)
    nbytes = alg_token_heads(wl, prefix is not None) * REF_BYTES_PER_TOKEN_HEAD[fmt]
    del cache, ws, out
    torch.cuda.empty_cache()
    return {"tokens_per_s": wl.total_tokens() / (ms_step * 1e-3), "ms_per_step": ms_step,
            "decode_kernel_ms": dec_ms, "bytes_per_token_head": REF_BYTES_PER_TOKEN_HEAD[fmt],
            "kv_gbs": nbytes / (dec_ms * 1e-3) / 1e9, "kv_frac": nbytes / (dec_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
            "flushed": {"tokens_per_s": wl.total_tokens() / (f_step * 1e-3), "ms_per_step": f_step,
                        "decode_kernel_ms": f_dec, "kv_gbs": nbytes / (f_dec * 1e-3) / 1e9,
                        "kv_frac": nbytes / (f_dec * 1e-3) / 1e9 / HBM_PEAK_GBS},
            "traffic": profiled_traffic(wl.name, fmt)}


def write_path(uq, args, dev, stream, flush):
    """Quantize-on-write (Algorithm 1, Write) on its own: a 65536-token bf16
    prefill of 8 KV heads into random pages, and a 1-token append for each of
    256 sequences through a page table. Algorithmic bytes of the prefill:
    the bf16 K and V rows read plus 136 B per token and KV head written."""
    import torch
    from paper_2606_20474_amd import workloads
    ww = workloads.WriteWorkload()
    data = ww.build(device=dev)
    kp, vp, pslots = data["prefill"]
    ka, va, aslots, pt, _ = data["append"]
    desc = uq.CacheDesc(num_kv_heads=ww.num_kv_heads, num_pages=ww.num_pages)
    codes, scales = desc.alloc_pools(dev)
    pslots = torch.as_tensor(pslots, device=dev)
    aslots = torch.as_tensor(aslots, device=dev)
    pt = torch.as_tensor(pt, device=dev)

    def prefill(ev_a=None, ev_b=None):
        if ev_a is not None:
            uq.time_next_launch(ev_a, ev_b)
        uq.quantize_kv(desc, kp, vp, pslots, codes, scales)

    def append(ev_a=None, ev_b=None):
        if ev_a is not None:
            uq.time_next_launch(ev_a, ev_b)
        uq.quantize_kv(desc, ka, va, aslots, codes, scales, page_table=pt)

    n = max(args.steps, 10)
    _, pre_ms = timed(prefill, n, 3, stream, flush=flush)
    _, pre_ms_b2b = timed(prefill, n, 3, stream)
    _, app_ms = timed(append, n, 3, stream)
    rd = 2 * kp.numel() * kp.element_size()
    wr = ww.prefill_tokens * ww.num_kv_heads * KV_BYTES_PER_TOKEN_HEAD
    gbs = (rd + wr) / (pre_ms * 1e-3) / 1e9
    # what this GPU moves for reads plus writes: torch's device-to-device
    # copy of 512 MiB, timed like the prefill (event pair around the launch,
    # after the flush); a reference point, not the roof the fraction uses
    src = torch.empty(512 << 20, dtype=torch.uint8, device=dev)
    dst = torch.empty_like(src)

    def copy(ev_a=None, ev_b=None):
        dst.copy_(src)
    copy_ms, _ = timed(copy, max(10, n // 4), 2, stream, flush=flush)
    copy_gbs = 2 * src.numel() / (copy_ms * 1e-3) / 1e9
    del src, dst
    return {"prefill_tokens": ww.prefill_tokens, "num_kv_heads": ww.num_kv_heads, "in_dtype": "bf16",
            "prefill_us": pre_ms * 1e3, "prefill_tokens_per_s": ww.prefill_tokens / (pre_ms * 1e-3),
            "prefill_bytes": rd + wr, "prefill_gbs": gbs, "prefill_frac": gbs / HBM_PEAK_GBS,
            "prefill_us_back_to_back": pre_ms_b2b * 1e3, "append_seqs": ww.append_seqs, "append_us": app_ms * 1e3,
            "copy_gbs": copy_gbs, "prefill_frac_of_copy": gbs / copy_gbs,
            "timing": "prefill and copy: 1 GiB written and read back before every launch, prefill by kernel events, "
                      "copy by an event pair around it; append: back to back"}


def achievable(uq, wl, desc, codes, scales, pt, ctx, part, alg_bytes, args, dev, stream, flush, prefix=None):
    """What this GPU delivers to the decode kernel's reads, timed like the
    kernel (flushed, kernel events): a plain stream of the launch's
    algorithmic bytes and of 4 GiB (uq_probe_stream_read), and the decode
    kernel's own page gather of this workload without its arithmetic
    (uq_probe_page_gather, or uq_probe_page_gather_cascade for a workload
    with a shared prefix: the kernel's own launch in its probe mode)."""
    import torch
    n = max(20, args.steps // 4)
    res = {}
    for name, nbytes in (("stream_same_bytes", alg_bytes), ("stream_4gib", 4 << 30)):
        buf = torch.zeros((nbytes + 15) // 16 * 16, dtype=torch.uint8, device=dev)
        sink = torch.empty(uq.PROBE_STREAM_BLOCKS, dtype=torch.int32, device=dev)

        def probe(ev_a=None, ev_b=None):
            if ev_a is not None:
                uq.time_next_launch(ev_a, ev_b)
            uq.probe_stream_read(buf, sink)
        _, ms = timed(probe, n, 3, stream, flush=flush)
        res[f"{name}_gbs"] = buf.numel() / (ms * 1e-3) / 1e9
        res[f"{name}_bytes"] = buf.numel()
        del buf, sink
        torch.cuda.empty_cache()
    # the decode kernel's own grid as a probe: plain (any head size) or the
    # cascade's, as the timed step runs it
    if prefix is None:
        sink = torch.empty(4 * max(1, -(-wl.max_context // part)) * wl.num_kv_heads * wl.batch, dtype=torch.int32,
                           device=dev)

        def gather(ev_a=None, ev_b=None):
            if ev_a is not None:
                uq.time_next_launch(ev_a, ev_b)
            uq.probe_page_gather(desc, wl.num_q_heads, codes, scales, pt, ctx, wl.max_context, part, sink)
    else:
        pws = torch.empty(uq.cascade_workspace_bytes(wl.num_kv_heads, wl.batch, wl.num_q_heads, wl.max_context,
                                                     prefix, part), dtype=torch.uint8, device=dev)
        sink = uq.probe_page_gather_cascade(desc, wl.num_q_heads, codes, scales, pt, ctx, wl.max_context, prefix,
                                            part, pws)

        def gather(ev_a=None, ev_b=None):
            if ev_a is not None:
                uq.time_next_launch(ev_a, ev_b)
            uq.probe_page_gather_cascade(desc, wl.num_q_heads, codes, scales, pt, ctx, wl.max_context, prefix, part,
                                         pws, sink)
    _, ms = timed(gather, n, 3, stream, flush=flush)
    res["page_gather_gbs"] = alg_bytes / (ms * 1e-3) / 1e9
    res["page_gather_ms"] = ms
    return res


def scaled_pv_ab(uq, wl, desc, codes, scales, q, pt, ctx, part, args, dev, stream, flush):
    """A/B of PV on the block-scaled FP4 x FP8 instruction
    (uq_decode_attention_scaled_pv) against the default BF16 PV
    (uq_decode_attention), both reading every sequence's whole context
    (no cascade, no fused write), kernel events on the partials launch,
    flushed like the headline kernel."""
    import torch
    ws = uq.alloc_workspace(desc, wl.batch, wl.num_q_heads, wl.max_context, part, dev)
    out = torch.empty((wl.batch, wl.num_q_heads, 128), dtype=torch.float32, device=dev)
    nbytes = wl.total_tokens() * wl.num_kv_heads * KV_BYTES_PER_TOKEN_HEAD
    n = max(20, args.steps // 4)
    res = {"kv_bytes_per_launch": nbytes}
    for name, fn in (("bf16_pv", uq.decode_attention), ("scaled_pv", uq.decode_attention_scaled_pv)):
        def step(ev_a=None, ev_b=None, fn=fn):
            if ev_a is not None:
                uq.time_next_launch(ev_a, ev_b)
            fn(desc, q, codes, scales, pt, ctx, wl.max_context, 1 / math.sqrt(128), part, workspace=ws, out=out)
        st, k = timed(step, n, 3, stream, flush=None if args.no_flush else flush)
        res[name] = {"kernel_ms": k, "kernel_gbs": nbytes / (k * 1e-3) / 1e9, "ms_per_step": st}
    res["scaled_over_bf16_kernel_ms"] = res["scaled_pv"]["kernel_ms"] / res["bf16_pv"]["kernel_ms"]
    del ws, out
    torch.cuda.empty_cache()
    return res


def cpu_baseline(wl, nseq, dev):
    """The oracle on `nseq` sequences of the workload (all their query heads,
    full contexts), timed on the host; KV tokens/s."""
    import oracle
    seqs = list(range(min(nseq, wl.batch)))
    maxp = wl.max_pages_per_seq
    pt = np.arange(len(seqs) * maxp, dtype=np.int32).reshape(len(seqs), maxp)
    pools = oracle.alloc_pools(len(seqs) * maxp, wl.num_kv_heads, head_dim=wl.head_dim)
    for i, b in enumerate(seqs):
        for key, lo, hi in wl.sequence_segments(b):
            k, v = wl.kv(key, lo, hi, device=dev)
            pos = np.arange(lo, hi, dtype=np.int64)
            slots = pt[i, pos // 16].astype(np.int64) * 16 + pos % 16
            oracle.quantize_kv(k.cpu().numpy(), v.cpu().numpy(), slots, len(seqs) * maxp, rotate_v=wl.rotate_v,
                               pools=pools)
    q = wl.q.numpy()[seqs]
    ctx = wl.context_lens[seqs]
    t0 = time.perf_counter()
    oracle.decode_attention(q, pools, pt, ctx, wl.num_kv_heads, 1 / math.sqrt(wl.head_dim), wl.rotate_v)
    dt = time.perf_counter() - t0
    toks = int(ctx.astype(np.int64).sum())
    return {"value": toks / dt, "unit": "tokens/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"{len(seqs)} of {wl.batch} sequences, all {wl.num_q_heads} query heads, "
                      f"{toks} context tokens; fp64 decode attention over the oracle's own FP4 cache; "
                      f"{dt:.2f} s wall on {oracle.num_threads()} threads ({dt * oracle.num_threads():.0f} "
                      f"thread-seconds)"}


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the library has no multi-GPU path.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2606_20474_amd import uq

    dev = torch.device("cuda:0")
    wl = make_workload(args.workload)
    part = wl.partition_tokens if args.partition < 0 else args.partition
    D = wl.head_dim
    desc = uq.CacheDesc(num_kv_heads=wl.num_kv_heads, num_pages=wl.num_pages, rotate_v=wl.rotate_v, head_dim=D)
    codes, scales = desc.alloc_pools(dev)
    fill_cache(uq, wl, desc, codes, scales, dev)
    progress(f"{wl.name}: FP4 cache written")
    if part == 0:
        part = uq.default_partition(desc, wl.batch, wl.num_q_heads, wl.max_context)

    q = wl.q.to(dev)
    pt = torch.as_tensor(wl.page_table, device=dev)
    ctx = torch.as_tensor(wl.context_lens, device=dev)
    prefix = None
    if wl.shared_prefix_tokens and not args.no_cascade:
        prefix = uq.SharedPrefix(torch.as_tensor(wl.prefix_pages.astype(np.int32), device=dev),
                                 torch.as_tensor(wl.prefix_lens(), device=dev), wl.shared_prefix_tokens)
        ws = torch.empty(uq.cascade_workspace_bytes(wl.num_kv_heads, wl.batch, wl.num_q_heads, wl.max_context, prefix,
                                                    part), dtype=torch.uint8, device=dev)
    else:
        ws = uq.alloc_workspace(desc, wl.batch, wl.num_q_heads, wl.max_context, part, dev)
    out = torch.empty((wl.batch, wl.num_q_heads, D), dtype=torch.float32, device=dev)
    # the step's new token of every sequence (written at its last position by the step)
    g = torch.Generator(device=dev).manual_seed(12345)
    k_new = torch.randn((wl.batch, wl.num_kv_heads, D), generator=g, device=dev)
    v_new = torch.randn((wl.batch, wl.num_kv_heads, D), generator=g, device=dev)
    last = wl.context_lens.astype(np.int64) - 1
    new_slots = torch.as_tensor(wl.page_table[np.arange(wl.batch), last // 16].astype(np.int64) * 16 + last % 16,
                                device=dev)
    scale = 1 / math.sqrt(D)
    stream = torch.cuda.current_stream()

    def step(ev_a=None, ev_b=None):
        if D != 128:
            # head sizes 64 and 256: the write of the new tokens is its own launch
            uq.quantize_kv(desc, k_new, v_new, new_slots, codes, scales)
        if ev_a is not None:
            uq.time_next_launch(ev_a, ev_b)
        if D != 128:
            uq.decode_partials(desc, q, codes, scales, pt, ctx, wl.max_context, scale, part, ws, out)
        elif prefix is None:
            uq.decode_step(desc, q, k_new, v_new, codes, scales, pt, ctx, wl.max_context, scale, part, ws, out,
                           partials_only=True)
        else:
            uq.decode_cascade(desc, q, codes, scales, pt, ctx, wl.max_context, prefix, scale, part, ws, out,
                              k_new=k_new, v_new=v_new, partials_only=True)
        if prefix is None:
            uq.decode_merge(desc, wl.batch, wl.num_q_heads, ctx, wl.max_context, part, ws, out)
        else:
            uq.decode_cascade_merge(desc, wl.batch, wl.num_q_heads, ctx, wl.max_context, prefix, part, ws, out)

    if args.calib_copy_mib > 0:
        n = args.calib_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty(n, dtype=torch.uint8, device=dev)
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    flush = make_flush(dev)
    ms_step, dec_ms_b2b = timed(step, args.steps, args.warmup, stream)
    if args.no_flush:
        f_step, dec_ms = ms_step, dec_ms_b2b
    else:
        f_step, dec_ms = timed(step, args.steps, args.warmup, stream, flush=flush)
    progress(f"FP4 step timed: {ms_step * 1e3:.1f} us back to back, {f_step * 1e3:.1f} us flushed")

    tokens = wl.total_tokens()
    kv_bytes = wl.kv_bytes_fp4()            # logical: every sequence's whole context
    alg_tokens = alg_token_heads(wl, prefix is not None) // wl.num_kv_heads
    alg_bytes = alg_tokens * wl.num_kv_heads * (KV_BYTES_PER_TOKEN_HEAD * D // 128)
    achieved = alg_bytes / (dec_ms * 1e-3) / 1e9
    ach = None if args.no_probes else achievable(uq, wl, desc, codes, scales, pt, ctx, part, alg_bytes, args, dev,
                                                 stream, flush, prefix)
    if ach is not None:
        progress("bandwidth probes timed")
    result = {
        "metric": "decode-attention KV tokens/s and achieved HBM GB/s (% of peak) at 32k context",
        "value": tokens / (ms_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp4-e2m1+ue8m0 kv, fp8-e4m3 q, fp32 accum",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": wl.batch, "num_q_heads": wl.num_q_heads,
                   "num_kv_heads": wl.num_kv_heads, "head_dim": D, "context": int(wl.max_context),
                   "page_size": 16, "partition_tokens": int(part), "parallelism": "single-gpu",
                   "shared_prefix_tokens": int(wl.shared_prefix_tokens), "cascade": prefix is not None},
        "hbm_gbs_step": kv_bytes / (ms_step * 1e-3) / 1e9,
        "hbm_frac_step": kv_bytes / (ms_step * 1e-3) / 1e9 / HBM_PEAK_GBS,
        "roofline": {"bound": "hbm", "kernel": "decode_kernel", "achieved": achieved, "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": achieved / HBM_PEAK_GBS, "traffic": profiled_traffic(wl.name),
                     "launch_ms": dec_ms, "bytes_per_launch": alg_bytes, "logical_bytes_per_launch": kv_bytes,
                     "timing": "kernel events (uq_time_next_launch), 1 GiB written and read back before every launch"
                               + (" (not: --no-flush)" if args.no_flush else ""),
                     "launch_ms_back_to_back": dec_ms_b2b,
                     "achieved_back_to_back": alg_bytes / (dec_ms_b2b * 1e-3) / 1e9},
        "flushed": {"ms_per_step": f_step, "tokens_per_s": tokens / (f_step * 1e-3),
                    "step_timing": "event pair around the step's launches, 1 GiB written and read back before every step"},
    }
    if ach is not None:
        result["achievable"] = ach
        if ach.get("page_gather_gbs"):
            result["roofline"]["achievable_gbs"] = ach["page_gather_gbs"]
            result["roofline"]["frac_of_achievable"] = achieved / ach["page_gather_gbs"]
    # the comparison caches exist at head size 128
    fmts = [f for f in args.comparators.split(",") if f and f != "none"] if D == 128 else []
    if fmts:
        comp = {}
        for fmt in fmts:
            if fmt not in REF_BYTES_PER_TOKEN_HEAD:
                sys.exit(f"unknown comparator {fmt!r}")
            comp[f"{fmt}_kv"] = comparator(uq, fmt, wl, part, q, pt, ctx, k_new, v_new, args, dev, stream, flush,
                                           prefix)
            progress(f"{fmt} comparator timed")
            comp[f"fp4_over_{fmt}_tokens_per_s"] = result["value"] / comp[f"{fmt}_kv"]["tokens_per_s"]
            comp[f"fp4_over_{fmt}_tokens_per_s_flushed"] = (result["flushed"]["tokens_per_s"]
                                                           / comp[f"{fmt}_kv"]["flushed"]["tokens_per_s"])
        result["comparators"] = comp
    if D == 128 and not args.no_scaled_pv:
        result["scaled_pv_ab"] = scaled_pv_ab(uq, wl, desc, codes, scales, q, pt, ctx, part, args, dev, stream,
                                              flush)
        progress("scaled-PV A/B timed")
    if not args.no_write_path:
        result["write_path"] = write_path(uq, args, dev, stream, flush)
        progress("write path timed")
    if not args.no_cpu_baseline:
        result["cpu_baseline"] = cpu_baseline(wl, args.cpu_sample_seqs, dev)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
