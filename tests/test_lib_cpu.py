"""Host-side checks of libuq that need no GPU: the library builds and loads,
exports every entry point include/uq.h declares, and rejects bad arguments
with the documented status before any HIP call."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def uq():
    from paper_2606_20474_amd import build
    if not os.path.exists(build.LIB):
        build.build()
    from paper_2606_20474_amd import uq as mod
    return mod


def header_functions():
    text = open(os.path.join(ROOT, "include", "uq.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(uq_[a-z0-9_]+)\s*\(", text)))


def test_exports_every_declared_symbol(uq):
    names = header_functions()
    assert len(names) >= 7
    for n in names:
        assert hasattr(uq.lib, n), n
    assert sorted(uq.EXPORTS) == names


def test_status_strings_are_total(uq):
    for s in range(5):
        assert uq.status_string(s).startswith("UQ_")
    assert uq.status_string(99) == "UQ_ERR_UNKNOWN"
    assert uq.lib.uq_version() >= 100


FAKE = ctypes.c_void_p(0x10000)   # aligned, never dereferenced: validation fails first or nothing is launched


def desc(**kw):
    from paper_2606_20474_amd.uq import uq_cache_desc
    d = dict(num_kv_heads=2, head_dim=128, page_size=16, group_size=32, num_pages=10, c=0.156, rotate_v=1)
    d.update(kw)
    return uq_cache_desc(**d)


def quantize(uq, d, num_tokens=4, stride=256, k=FAKE, pt=None, num_seqs=0, mpps=0, dtype=1, slots=FAKE):
    return uq.lib.uq_quantize_kv(ctypes.byref(d) if d is not None else None, k, FAKE, dtype, num_tokens, stride, pt,
                                 num_seqs, mpps, slots, FAKE, FAKE, None)


def test_quantize_validation(uq):
    E = uq
    assert quantize(uq, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(head_dim=96)) == E.UQ_ERR_UNSUPPORTED
    assert quantize(uq, desc(page_size=32)) == E.UQ_ERR_UNSUPPORTED
    assert quantize(uq, desc(group_size=16)) == E.UQ_ERR_UNSUPPORTED
    assert quantize(uq, desc(c=0.0)) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(c=float("nan"))) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(num_kv_heads=0)) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(num_pages=0)) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(), num_tokens=-1) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(), k=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(), slots=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(), stride=255) == E.UQ_ERR_INVALID_ARGUMENT      # below Hkv * 128
    assert quantize(uq, desc(), stride=260) == E.UQ_ERR_INVALID_ARGUMENT      # not 16-byte aligned rows
    assert quantize(uq, desc(), k=ctypes.c_void_p(0x10004)) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(), dtype=3) == E.UQ_ERR_UNSUPPORTED
    assert quantize(uq, desc(), pt=FAKE, num_seqs=0, mpps=4) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(), pt=FAKE, num_seqs=2, mpps=0) == E.UQ_ERR_INVALID_ARGUMENT
    assert quantize(uq, desc(), num_tokens=0) == E.UQ_OK                     # no-op, nothing launched


def decode(uq, d, q=FAKE, qdt=0, B=2, Hq=4, mpps=4, maxctx=64, scale=0.1, part=0, ws=FAKE, wsb=1 << 30, out=FAKE,
           odt=0, ctx=FAKE, pt=FAKE):
    return uq.lib.uq_decode_attention(ctypes.byref(d) if d is not None else None, q, qdt, B, Hq, FAKE, FAKE, pt, mpps,
                                      ctx, maxctx, scale, part, ws, wsb, out, odt, None)


def test_decode_validation(uq):
    E = uq
    assert decode(uq, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(head_dim=96)) == E.UQ_ERR_UNSUPPORTED
    assert decode(uq, desc(), Hq=3) == E.UQ_ERR_INVALID_ARGUMENT               # Hq % Hkv
    assert decode(uq, desc(), Hq=34) == E.UQ_ERR_UNSUPPORTED                   # 17 query heads per kv head
    assert decode(uq, desc(), B=0) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), maxctx=65) == E.UQ_ERR_INVALID_ARGUMENT          # > max_pages_per_seq * 16
    assert decode(uq, desc(), maxctx=-1) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), part=40) == E.UQ_ERR_INVALID_ARGUMENT            # not whole pages (16 tokens)
    assert decode(uq, desc(), scale=float("inf")) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), scale=0.0) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), scale=-0.1) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), q=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), pt=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), ctx=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), out=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), qdt=7) == E.UQ_ERR_UNSUPPORTED
    assert decode(uq, desc(), odt=3) == E.UQ_ERR_UNSUPPORTED
    assert decode(uq, desc(), ws=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode(uq, desc(), wsb=16) == E.UQ_ERR_WORKSPACE_TOO_SMALL
    assert decode(uq, desc(), q=ctypes.c_void_p(0x10008)) == E.UQ_ERR_INVALID_ARGUMENT
    # partitions x kv heads x sequences beyond one 2^31 linear grid
    big = desc(num_kv_heads=65535)
    assert decode(uq, big, B=65535, Hq=65535, part=32, wsb=1 << 62) == E.UQ_ERR_UNSUPPORTED


def decode_noalloc(uq, d, q=FAKE, qdt=0, B=2, Hq=4, mpps=4, maxctx=64, scale=0.1, part=0, out=FAKE, odt=0, ctx=FAKE,
                   pt=FAKE):
    return uq.lib.uq_decode_attention_noalloc(ctypes.byref(d) if d is not None else None, q, qdt, B, Hq, FAKE, FAKE,
                                              pt, mpps, ctx, maxctx, scale, part, out, odt, None)


def test_scaled_pv_validation(uq):
    """The prototype takes the decode call's checks, head size 128 only and
    partitions of whole page pairs (32 tokens)."""
    E = uq
    def call(d, part=0):
        return uq.lib.uq_decode_attention_scaled_pv(ctypes.byref(d), FAKE, 0, 2, 4, FAKE, FAKE, FAKE, 4, FAKE, 64,
                                                    0.1, part, FAKE, 1 << 30, FAKE, 0, None)
    assert call(desc(), part=40) == E.UQ_ERR_INVALID_ARGUMENT
    assert call(desc(), part=48) == E.UQ_ERR_INVALID_ARGUMENT
    assert call(desc(head_dim=64)) == E.UQ_ERR_UNSUPPORTED


def test_decode_noalloc_validation(uq):
    """The no-allocation decode makes uq_decode_attention's host checks, and
    refuses a call whose partials exceed its device array, before any HIP
    call (so before it looks the array up)."""
    E = uq
    assert decode_noalloc(uq, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode_noalloc(uq, desc(head_dim=96)) == E.UQ_ERR_UNSUPPORTED
    assert decode_noalloc(uq, desc(), Hq=3) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode_noalloc(uq, desc(), maxctx=65) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode_noalloc(uq, desc(), part=40) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode_noalloc(uq, desc(), q=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode_noalloc(uq, desc(), out=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert decode_noalloc(uq, desc(), odt=3) == E.UQ_ERR_UNSUPPORTED
    # 256 sequences x 64 query heads x 32 partitions of 4096 tokens (128k
    # contexts): 273 MB of partials, beyond the array
    from paper_2606_20474_amd.uq import CacheDesc
    big = desc(num_kv_heads=8, num_pages=1 << 21)
    need = uq.workspace_bytes(CacheDesc(num_kv_heads=8, num_pages=1 << 21), 256, 64, 131072, 4096)
    assert need > uq.NOALLOC_SCRATCH_BYTES
    assert decode_noalloc(uq, big, B=256, Hq=64, mpps=8192, maxctx=131072, part=4096) == E.UQ_ERR_WORKSPACE_TOO_SMALL
    # the Qwen3-235B-like layer's partials (4.3 MB at the default partition) fit
    qwen = CacheDesc(num_kv_heads=4, num_pages=65536)
    assert uq.workspace_bytes(qwen, 32, 64, 32768, 0) <= uq.NOALLOC_SCRATCH_BYTES
    text = open(os.path.join(ROOT, "include", "uq.h")).read()
    assert re.search(r"#define UQ_NOALLOC_SCRATCH_BYTES \(\(size_t\)32 << 20\)", text)
    assert uq.NOALLOC_SCRATCH_BYTES == 32 << 20


def test_workspace_and_partition_sizes(uq):
    from paper_2606_20474_amd.uq import CacheDesc
    d = CacheDesc(num_kv_heads=4, num_pages=65536)
    p = uq.default_partition(d, 32, 64, 32768)
    assert p % 32 == 0 and 1024 <= p <= 16384
    np_ = -(-32768 // p)
    assert uq.workspace_bytes(d, 32, 64, 32768, 0) == 32 * 64 * np_ * 130 * 4
    assert uq.workspace_bytes(d, 32, 64, 32768, 4096) == 32 * 64 * 8 * 130 * 4
    assert uq.workspace_bytes(d, 32, 63, 32768, 4096) == 0   # invalid: returns 0
    assert uq.workspace_bytes(d, 1, 4, 0, 0) == 4 * 1 * 130 * 4


def rdesc(**kw):
    from paper_2606_20474_amd.uq import uq_ref_cache_desc
    d = dict(num_kv_heads=2, head_dim=128, page_size=16, format=1, num_pages=10, k_scale=0.5, v_scale=0.25)
    d.update(kw)
    return uq_ref_cache_desc(**d)


def test_ref_cache_sizes_and_validation(uq):
    E = uq
    lib = uq.lib
    assert lib.uq_ref_cache_bytes(ctypes.byref(rdesc())) == 10 * 2 * 2 * 2048
    assert lib.uq_ref_cache_bytes(ctypes.byref(rdesc(format=2))) == 10 * 2 * 2 * 4096
    assert lib.uq_ref_cache_bytes(ctypes.byref(rdesc(format=3))) == 0              # TQ4 without a codebook
    assert lib.uq_ref_cache_bytes(ctypes.byref(rdesc(format=4))) == 0
    assert lib.uq_ref_cache_bytes(ctypes.byref(rdesc(k_scale=0.0))) == 0
    assert lib.uq_ref_cache_bytes(ctypes.byref(rdesc(format=2, k_scale=0.0))) > 0   # scales unused for BF16
    assert lib.uq_ref_cache_bytes(None) == 0

    def write(d, **kw):
        a = dict(k=FAKE, dtype=1, num_tokens=4, stride=256, pt=None, num_seqs=0, mpps=0, cache=FAKE)
        a.update(kw)
        return lib.uq_ref_write_kv(ctypes.byref(d) if d is not None else None, a["k"], FAKE, a["dtype"],
                                   a["num_tokens"], a["stride"], a["pt"], a["num_seqs"], a["mpps"], FAKE,
                                   a["cache"], None)

    assert write(None) == E.UQ_ERR_INVALID_ARGUMENT
    assert write(rdesc(format=0)) == E.UQ_ERR_UNSUPPORTED
    assert write(rdesc(head_dim=64)) == E.UQ_ERR_UNSUPPORTED
    assert write(rdesc(v_scale=float("inf"))) == E.UQ_ERR_INVALID_ARGUMENT
    assert write(rdesc(k_scale=-1.0)) == E.UQ_ERR_INVALID_ARGUMENT
    assert write(rdesc(), dtype=3) == E.UQ_ERR_UNSUPPORTED
    assert write(rdesc(), cache=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert write(rdesc(), cache=ctypes.c_void_p(0x10008)) == E.UQ_ERR_INVALID_ARGUMENT
    assert write(rdesc(), stride=128) == E.UQ_ERR_INVALID_ARGUMENT
    assert write(rdesc(), pt=FAKE, num_seqs=1, mpps=0) == E.UQ_ERR_INVALID_ARGUMENT
    assert write(rdesc(), num_tokens=0) == E.UQ_OK

    def rdecode(d, **kw):
        a = dict(q=FAKE, qdt=0, B=2, Hq=4, mpps=4, ctx=FAKE, maxctx=64, scale=0.1, part=0, ws=FAKE, wsb=1 << 30,
                 out=FAKE, odt=0)
        a.update(kw)
        return lib.uq_ref_decode_attention(ctypes.byref(d), a["q"], a["qdt"], a["B"], a["Hq"], FAKE, FAKE, a["mpps"],
                                           a["ctx"], a["maxctx"], a["scale"], a["part"], a["ws"], a["wsb"],
                                           a["out"], a["odt"], None)

    assert rdecode(rdesc(), qdt=3) == E.UQ_ERR_UNSUPPORTED          # the query is never pre-cast here
    assert rdecode(rdesc(), Hq=3) == E.UQ_ERR_INVALID_ARGUMENT
    assert rdecode(rdesc(), maxctx=65) == E.UQ_ERR_INVALID_ARGUMENT
    assert rdecode(rdesc(), part=24) == E.UQ_ERR_INVALID_ARGUMENT   # not whole pages
    assert rdecode(rdesc(), scale=0.0) == E.UQ_ERR_INVALID_ARGUMENT
    assert rdecode(rdesc(), wsb=16) == E.UQ_ERR_WORKSPACE_TOO_SMALL
    assert rdecode(rdesc(format=5)) == E.UQ_ERR_UNSUPPORTED
    assert rdecode(rdesc(), out=None) == E.UQ_ERR_INVALID_ARGUMENT
    # the same workspace formula as the FP4 cache
    from paper_2606_20474_amd.uq import CacheDesc
    d4 = CacheDesc(num_kv_heads=2, num_pages=10)
    assert uq.ref_workspace_bytes(uq.RefCacheDesc(2, 10, "bf16"), 32, 64, 32768, 0) == \
        uq.workspace_bytes(d4, 32, 64, 32768, 0)
    assert lib.uq_ref_decode_merge(ctypes.byref(rdesc()), 2, 4, None, 64, 0, FAKE, 1 << 30, FAKE, 0, None) == \
        E.UQ_ERR_INVALID_ARGUMENT


def test_decode_step_validation(uq):
    E = uq
    lib = uq.lib

    def step(d, **kw):
        a = dict(q=FAKE, kn=FAKE, vn=FAKE, ndt=0, B=2, Hq=4, ctx=FAKE, maxctx=64, scale=0.1, wsb=1 << 30)
        a.update(kw)
        return lib.uq_decode_step(ctypes.byref(d), a["q"], 0, a["kn"], a["vn"], a["ndt"], a["B"], a["Hq"], FAKE, FAKE,
                                  FAKE, 4, a["ctx"], a["maxctx"], a["scale"], 0, FAKE, a["wsb"], FAKE, 0, None)

    assert step(desc(), kn=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert step(desc(), vn=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert step(desc(), kn=ctypes.c_void_p(0x10004)) == E.UQ_ERR_INVALID_ARGUMENT
    assert step(desc(), ndt=3) == E.UQ_ERR_UNSUPPORTED
    assert step(desc(), Hq=3) == E.UQ_ERR_INVALID_ARGUMENT
    assert step(desc(), wsb=16) == E.UQ_ERR_WORKSPACE_TOO_SMALL
    assert step(desc(head_dim=64)) == E.UQ_ERR_UNSUPPORTED
    r = lib.uq_ref_decode_step(ctypes.byref(rdesc()), FAKE, 0, None, FAKE, 0, 2, 4, FAKE, FAKE, 4, FAKE, 64, 0.1, 0,
                               FAKE, 1 << 30, FAKE, 0, None)
    assert r == E.UQ_ERR_INVALID_ARGUMENT
    r = lib.uq_ref_decode_step_partials(ctypes.byref(rdesc()), FAKE, 0, FAKE, FAKE, 3, 2, 4, FAKE, FAKE, 4, FAKE, 64,
                                        0.1, 0, FAKE, 1 << 30, FAKE, 0, None)
    assert r == E.UQ_ERR_UNSUPPORTED


def test_cascade_validation(uq):
    E = uq
    lib = uq.lib
    from paper_2606_20474_amd.uq import uq_shared_prefix

    def pre(**kw):
        a = dict(pages=0x10000, lens=0x10000, num_tokens=64, partition_tokens=0)
        a.update(kw)
        return uq_shared_prefix(**a)

    def casc(sp, **kw):
        a = dict(kn=None, vn=None, wsb=1 << 30)
        a.update(kw)
        return lib.uq_decode_cascade(ctypes.byref(desc()), FAKE, 0, a["kn"], a["vn"], 0, 2, 4, FAKE, FAKE, FAKE, 4,
                                     FAKE, 64, ctypes.byref(sp) if sp is not None else None, 0.1, 0, FAKE,
                                     a["wsb"], FAKE, 0, None)

    assert casc(None) == E.UQ_ERR_INVALID_ARGUMENT
    assert casc(pre(pages=None)) == E.UQ_ERR_INVALID_ARGUMENT
    assert casc(pre(lens=None)) == E.UQ_ERR_INVALID_ARGUMENT
    assert casc(pre(num_tokens=40)) == E.UQ_ERR_INVALID_ARGUMENT      # not whole pages
    assert casc(pre(num_tokens=0)) == E.UQ_ERR_INVALID_ARGUMENT
    assert casc(pre(partition_tokens=48)) == E.UQ_ERR_INVALID_ARGUMENT
    assert casc(pre(), kn=FAKE) == E.UQ_ERR_INVALID_ARGUMENT          # k_new without v_new
    assert casc(pre(), wsb=16) == E.UQ_ERR_WORKSPACE_TOO_SMALL
    sp = pre(partition_tokens=32)
    # 64 context tokens in partitions of 32 -> 2 slots, plus 2 prefix partitions of 32
    plain = uq.workspace_bytes(__import__("paper_2606_20474_amd.uq", fromlist=["CacheDesc"]).CacheDesc(2, 10), 2, 4,
                               64, 32)
    # twice the partial rows, then the dispatch list: 16 bytes per context row
    # (2 partitions x 2 sequences) and per prefix row (1 column chunk x 2
    # prefix partitions)
    assert lib.uq_decode_cascade_workspace_bytes(2, 2, 4, 64, 32, ctypes.byref(sp)) == plain * 2 + (4 + 2) * 16
    assert lib.uq_decode_cascade_workspace_bytes(2, 2, 3, 64, 32, ctypes.byref(sp)) == 0
    r = lib.uq_ref_decode_cascade(ctypes.byref(rdesc()), FAKE, 0, None, None, 0, 2, 4, FAKE, FAKE, 4, FAKE, 64,
                                  None, 0.1, 0, FAKE, 1 << 30, FAKE, 0, None)
    assert r == E.UQ_ERR_INVALID_ARGUMENT
    r = lib.uq_decode_cascade_merge(ctypes.byref(desc()), 2, 4, FAKE, 64, ctypes.byref(pre(num_tokens=8)), 0, FAKE,
                                    1 << 30, FAKE, 0, None)
    assert r == E.UQ_ERR_INVALID_ARGUMENT


def test_quantize_error_validation(uq):
    E = uq
    f = uq.lib.uq_quantize_error
    assert f(FAKE, E.UQ_FP8_E4M3, 4, 128, 1, 1, 1, FAKE, FAKE, None) == E.UQ_ERR_UNSUPPORTED
    assert f(None, E.UQ_F32, 4, 128, 1, 1, 1, FAKE, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert f(None, E.UQ_F32, 0, 128, 1, 1, 1, FAKE, FAKE, None) == E.UQ_OK
    assert f(FAKE, E.UQ_F32, 4, 128, 1, 1, 1, None, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert f(FAKE, E.UQ_F32, 4, 128, 1, 1, 1, FAKE, None, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert f(FAKE, E.UQ_F32, -1, 128, 1, 1, 1, FAKE, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert f(FAKE, E.UQ_F32, 4, 127, 1, 1, 1, FAKE, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert f(FAKE, E.UQ_F32, 4, 130, 1, 1, 1, FAKE, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert f(FAKE, E.UQ_BF16, 4, 132, 1, 1, 1, FAKE, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert f(ctypes.c_void_p(0x10008), E.UQ_F32, 4, 128, 1, 1, 1, FAKE, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert f(FAKE, E.UQ_F32, 4, 128, 1, 1, -1, FAKE, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    # nothing to do: no launch
    assert f(FAKE, E.UQ_F32, 0, 128, 1, 1, 3, FAKE, FAKE, None) == E.UQ_OK
    assert f(FAKE, E.UQ_BF16, 4, 136, 1, 0, 0, FAKE, FAKE, None) == E.UQ_OK


def test_tq4_codebook_validation(uq):
    """The Ultra-TQ descriptor needs 16 finite levels, strictly ascending once
    rounded to BF16; the cache block is 2368 bytes per page and kv head."""
    import numpy as np
    E = uq
    lib = uq.lib
    from paper_2606_20474_amd.codebook import default_tq_codebook

    def tq(cb):
        cb = np.ascontiguousarray(cb, np.float32)
        d = rdesc(format=3, k_scale=0.0, v_scale=float("nan"))    # the scales are ignored
        d.codebook = ctypes.c_void_p(cb.ctypes.data)
        return d, cb

    good = default_tq_codebook(128)
    d, keep = tq(good)
    assert lib.uq_ref_cache_bytes(ctypes.byref(d)) == 10 * 2 * 2368
    bad = [good[::-1], np.where(np.arange(16) == 3, np.nan, good), np.linspace(1.0, 1.0 + 15 * 2 ** -10, 16),
           np.where(np.arange(16) == 15, np.inf, good)]
    for cb in bad:
        d, keep = tq(cb)
        assert lib.uq_ref_cache_bytes(ctypes.byref(d)) == 0
        assert lib.uq_ref_write_kv(ctypes.byref(d), FAKE, FAKE, 1, 4, 256, None, 0, 0, FAKE, FAKE, None) == \
            E.UQ_ERR_INVALID_ARGUMENT
    assert uq.RefCacheDesc(2, 10, "tq4").cache_bytes() == 10 * 2 * 2368


def test_head_sizes_64_and_256(uq):
    """Head sizes 64 and 256 pass validation for write and decode; the
    decode step, cascade, the FP8-query form and uq_prepare_query are
    head-size-128 calls (UNSUPPORTED otherwise).  Workspace rows hold d + 2
    floats."""
    E = uq
    lib = uq.lib
    for d in (64, 256):
        # validation passes, then the launch fails for want of a GPU
        assert quantize(uq, desc(head_dim=d), stride=2 * d) == E.UQ_ERR_HIP
        assert quantize(uq, desc(head_dim=d), stride=2 * d - 8) == E.UQ_ERR_INVALID_ARGUMENT
        assert decode(uq, desc(head_dim=d)) == E.UQ_ERR_HIP
        assert decode(uq, desc(head_dim=d), qdt=3) == E.UQ_ERR_UNSUPPORTED
        assert lib.uq_prepare_query(ctypes.byref(desc(head_dim=d)), FAKE, 0, 4, FAKE, None) == E.UQ_ERR_UNSUPPORTED
        dd = desc(head_dim=d)
        w = lib.uq_decode_workspace_bytes(ctypes.byref(dd), 2, 4, 64, 32)
        w128 = lib.uq_decode_workspace_bytes(ctypes.byref(desc()), 2, 4, 64, 32)
        assert w == 2 * 4 * 2 * (d + 2) * 4 and w128 == 2 * 4 * 2 * 130 * 4
        from paper_2606_20474_amd.uq import uq_shared_prefix
        sp = uq_shared_prefix(0x10000, 0x10000, 64, 0)
        r = lib.uq_decode_cascade(ctypes.byref(dd), FAKE, 0, None, None, 0, 2, 4, FAKE, FAKE, FAKE, 4, FAKE, 64,
                                  ctypes.byref(sp), 0.1, 0, FAKE, 1 << 30, FAKE, 0, None)
        assert r == E.UQ_ERR_UNSUPPORTED
    cd = uq.CacheDesc(num_kv_heads=2, num_pages=10, head_dim=64)
    assert cd.codes_bytes() == 10 * 2 * 2 * 512 and cd.scales_bytes() == 10 * 2 * 2 * 32


def test_time_next_launch_validation(uq):
    """One event without the other is rejected; NULL, NULL clears (no HIP call)."""
    lib = uq.lib
    assert lib.uq_time_next_launch(FAKE, None) == uq.UQ_ERR_INVALID_ARGUMENT
    assert lib.uq_time_next_launch(None, FAKE) == uq.UQ_ERR_INVALID_ARGUMENT
    assert lib.uq_time_next_launch(None, None) == uq.UQ_OK


def test_default_partition_counts_blocks(uq):
    """The default partition is the longest (1024..16384) that still gives the
    256 CUs two blocks each, counting one block per KV head, or per pair of
    KV heads where head size 64 runs two per block (G <= 8, even KV heads)."""
    from paper_2606_20474_amd.uq import CacheDesc

    def pick(units, ctx):
        part = 16384
        while part > 1024 and units * -(-ctx // part) < 512:
            part //= 2
        return part

    for hd, hkv, hq, B, ctx in [(128, 4, 64, 32, 32768), (128, 8, 64, 256, 131072), (128, 8, 48, 64, 131072),
                                (64, 8, 64, 32, 32768), (64, 8, 128, 32, 32768), (64, 3, 24, 32, 32768),
                                (256, 8, 64, 32, 32768), (64, 2, 2, 1, 4096)]:
        d = CacheDesc(num_kv_heads=hkv, num_pages=16, head_dim=hd)
        paired = hd == 64 and hkv % 2 == 0 and hq <= 8 * hkv
        want = pick(B * (hkv // 2 if paired else hkv), ctx)
        assert uq.default_partition(d, B, hq, ctx) == want, (hd, hkv, hq, B, ctx)
        # the workspace follows the same pick
        assert uq.workspace_bytes(d, B, hq, ctx, 0) == uq.workspace_bytes(d, B, hq, ctx, want)


def test_probe_validation(uq):
    """The measurement probes check their arguments before any HIP call."""
    E = uq
    L = uq.lib
    assert L.uq_probe_stream_read(None, 1 << 20, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert L.uq_probe_stream_read(FAKE, 0, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert L.uq_probe_stream_read(FAKE, 1000, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT       # not 16-byte words
    assert L.uq_probe_stream_read(ctypes.c_void_p(0x10008), 1 << 20, FAKE, None) == E.UQ_ERR_INVALID_ARGUMENT
    assert L.uq_probe_stream_read(FAKE, 1 << 20, None, None) == E.UQ_ERR_INVALID_ARGUMENT

    def gather(d, B=2, Hq=4, mpps=4, maxctx=64, part=32, sink_words=1 << 20, pt=FAKE):
        return L.uq_probe_page_gather(ctypes.byref(d), B, Hq, FAKE, FAKE, pt, mpps, FAKE, maxctx, part, FAKE,
                                      sink_words, None)
    assert gather(desc(head_dim=96)) == E.UQ_ERR_UNSUPPORTED
    assert gather(desc(), Hq=3) == E.UQ_ERR_INVALID_ARGUMENT
    assert gather(desc(), maxctx=65) == E.UQ_ERR_INVALID_ARGUMENT
    assert gather(desc(), pt=None) == E.UQ_ERR_INVALID_ARGUMENT
    # 2 partitions x 2 kv heads x 2 sequences x 4 waves = 32 words
    assert gather(desc(), sink_words=31) == E.UQ_ERR_WORKSPACE_TOO_SMALL
    # head size 64 at group size 2: two kv heads per block, 16 words; a
    # valid call reaches the launch (a HIP error without a GPU)
    assert gather(desc(head_dim=64), sink_words=15) == E.UQ_ERR_WORKSPACE_TOO_SMALL
    assert gather(desc(head_dim=64), sink_words=16) == E.UQ_ERR_HIP

    from paper_2606_20474_amd.uq import uq_shared_prefix

    def cgather(sp, head_dim=128, sink_words=1 << 20, wsb=1 << 30):
        return L.uq_probe_page_gather_cascade(ctypes.byref(desc(head_dim=head_dim)), 2, 4, FAKE, FAKE, FAKE, 4, FAKE,
                                              64, ctypes.byref(sp) if sp is not None else None, 32, FAKE, wsb, FAKE,
                                              sink_words, None)
    sp = uq_shared_prefix(0x10000, 0x10000, 64, 32)
    assert cgather(None) == E.UQ_ERR_INVALID_ARGUMENT
    assert cgather(uq_shared_prefix(0x10000, 0x10000, 40, 0)) == E.UQ_ERR_INVALID_ARGUMENT
    assert cgather(sp, head_dim=64) == E.UQ_ERR_UNSUPPORTED
    assert cgather(sp, wsb=16) == E.UQ_ERR_WORKSPACE_TOO_SMALL
    # 2 context partitions x 2 kv heads x 2 sequences + 2 kv heads x 1 column
    # chunk x 2 prefix partitions = 12 blocks of 4 waves
    assert cgather(sp, sink_words=47) == E.UQ_ERR_WORKSPACE_TOO_SMALL
    assert cgather(sp, sink_words=48) == E.UQ_ERR_HIP

    def mfma(kind=0, a=FAKE, b=FAKE, sa=FAKE, sb=FAKE, n=1, d=FAKE):
        return L.uq_probe_mfma(kind, a, b, sa, sb, n, d, None)
    assert mfma(kind=4) == E.UQ_ERR_INVALID_ARGUMENT
    assert mfma(kind=-1) == E.UQ_ERR_INVALID_ARGUMENT
    assert mfma(n=0) == E.UQ_ERR_INVALID_ARGUMENT
    assert mfma(n=65536) == E.UQ_ERR_INVALID_ARGUMENT
    assert mfma(a=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert mfma(sa=None) == E.UQ_ERR_INVALID_ARGUMENT
    assert mfma(d=ctypes.c_void_p(0x10004)) == E.UQ_ERR_INVALID_ARGUMENT
