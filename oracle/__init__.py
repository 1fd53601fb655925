"""CPU oracle for the UltraQuant FP4 KV-cache path (test infrastructure).

Only the test suite, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg
of ``bench.py`` may import this package.  The product library never does.
The arithmetic lives in ``uq_oracle.c`` (plain C, fp64 attention); this
module only marshals numpy arrays through ctypes.  See the header of
``uq_oracle.c`` for what each function follows in the paper and for the
readings taken where the paper is silent.
"""
import ctypes
import os

import numpy as np

from . import build as _build

HEAD_DIM = 128
PAGE_SIZE = 16
TILE_CODES = 1024
TILE_SCALES = 64
C_DEFAULT = 0.156

_lib = None


def lib():
    """Load ``liboracle.so``, compiling it first if it is not there.  The
    environment variable UQ_ORACLE_LIB names another build of the same
    source instead (the planted-mistake test loads deliberately broken
    copies that way, in subprocesses of its own)."""
    global _lib
    if _lib is None:
        path = os.environ.get("UQ_ORACLE_LIB")
        if path:
            if not os.path.exists(path):
                raise FileNotFoundError(f"UQ_ORACLE_LIB={path} does not exist")
        else:
            path = _build.LIB
            if not os.path.exists(path):
                _build.build()
        L = ctypes.CDLL(path)
        vp, i64, i32, f32, f64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_double
        L.uqo_num_threads.restype = i32
        L.uqo_wht128_f32.argtypes = [vp, i64]
        L.uqo_wht128_f64.argtypes = [vp, vp]
        L.uqo_wht_f32.argtypes = [vp, i64, i32]
        L.uqo_wht_f64.argtypes = [vp, vp, i32]
        L.uqo_prepare_query_d.argtypes = [vp, i64, vp, i32]
        L.uqo_quantize_vector_d.argtypes = [vp, i32, f32, i32, vp, vp]
        L.uqo_quantize_vectors_d.argtypes = [vp, i64, i32, f32, i32, vp, vp]
        L.uqo_quantize_kv_d.argtypes = [vp, vp, i64, i32, i64, vp, i64, f32, i32, vp, vp, i32]
        L.uqo_quantize_kv_d.restype = i64
        L.uqo_load_vector_d.argtypes = [vp, vp, i32, i64, i32, i32, i32, vp, vp, i32]
        L.uqo_dequant_vector_d.argtypes = [vp, vp, i32, i64, i32, i32, i32, vp, i32]
        L.uqo_decode_attention_d.argtypes = [vp, i32, i32, i32, vp, vp, vp, i32, vp, f64, i32, vp, i32]
        L.uqo_scale_exponent.argtypes = [f32, f32]
        L.uqo_scale_exponent.restype = i32
        L.uqo_e2m1_encode.argtypes = [f32, i32]
        L.uqo_e2m1_encode.restype = ctypes.c_uint8
        L.uqo_e2m1_value.argtypes = [ctypes.c_uint8, i32]
        L.uqo_e2m1_value.restype = f64
        L.uqo_e4m3_encode.argtypes = [f32]
        L.uqo_e4m3_encode.restype = ctypes.c_uint8
        L.uqo_e4m3_value.argtypes = [ctypes.c_uint8]
        L.uqo_e4m3_value.restype = f64
        L.uqo_prepare_query.argtypes = [vp, i64, vp]
        L.uqo_quantize_vector.argtypes = [vp, f32, i32, vp, vp]
        L.uqo_quantize_vectors.argtypes = [vp, i64, f32, i32, vp, vp]
        L.uqo_quantize_kv.argtypes = [vp, vp, i64, i32, i64, vp, i64, f32, i32, vp, vp]
        L.uqo_quantize_kv.restype = i64
        L.uqo_load_vector.argtypes = [vp, vp, i32, i64, i32, i32, i32, vp, vp]
        L.uqo_dequant_vector.argtypes = [vp, vp, i32, i64, i32, i32, i32, vp]
        L.uqo_decode_attention.argtypes = [vp, i32, i32, i32, vp, vp, vp, i32, vp, f64, i32, vp]
        L.uqo_quantize_error.argtypes = [vp, i64, i32, i32, i32, vp, vp]
        L.uqo_bf16_rne.argtypes = [f32]
        L.uqo_bf16_rne.restype = f32
        L.uqo_tq4_encode_vector.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp]
        L.uqo_tq4_norm.argtypes = [vp]
        L.uqo_tq4_norm.restype = ctypes.c_float
        L.uqo_tq4_index.argtypes = [ctypes.c_float, ctypes.c_float, vp]
        L.uqo_tq4_index.restype = i32
        L.uqo_tq4_write.argtypes = [vp, vp, i64, i32, i64, vp, i64, vp, vp]
        L.uqo_tq4_write.restype = i64
        L.uqo_tq4_load.argtypes = [vp, i32, i64, i32, i32, vp, vp, vp, vp, vp]
        L.uqo_tq4_dequant.argtypes = [vp, i32, i64, i32, i32, vp, vp, vp]
        L.uqo_tq4_decode_attention.argtypes = [vp, i32, i32, i32, vp, vp, i32, vp, f64, vp, vp]
        _lib = L
    return _lib


def _ptr(a):
    return ctypes.c_void_p(a.ctypes.data)


def _f32(x):
    return np.ascontiguousarray(x, dtype=np.float32)


def num_threads():
    """Threads the oracle's OpenMP loops run on."""
    return int(lib().uqo_num_threads())


HEAD_DIMS = (64, 128, 256)


def _dim(d):
    d = int(d)
    assert d in HEAD_DIMS, d
    return d


def wht_f32(x):
    """fp32 butterfly rotation R x of each vector along the last axis
    (64, 128 or 256 channels; reading R1)."""
    y = _f32(x).copy()
    d = _dim(y.shape[-1])
    lib().uqo_wht_f32(_ptr(y), y.size // d, d)
    return y


def wht_f64(x):
    """Exact fp64 rotation H x / sqrt(d) of one vector."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    d = _dim(x.size)
    y = np.empty(d, np.float64)
    lib().uqo_wht_f64(_ptr(x), _ptr(y), d)
    return y


def wht128_f32(x):
    """fp32 butterfly rotation R x of each 128-vector (reading R1)."""
    assert np.shape(x)[-1] == HEAD_DIM
    return wht_f32(x)


def wht128_f64(x):
    """Exact fp64 rotation H x / sqrt(128) of one 128-vector."""
    assert np.size(x) == HEAD_DIM
    return wht_f64(x)


def scale_exponent(m, c=C_DEFAULT):
    return int(lib().uqo_scale_exponent(float(np.float32(m)), float(np.float32(c))))


def e2m1_encode(x, E):
    return int(lib().uqo_e2m1_encode(float(np.float32(x)), int(E)))


def e2m1_value(code, scale_byte):
    return float(lib().uqo_e2m1_value(int(code), int(scale_byte)))


def e4m3_encode(x):
    return int(lib().uqo_e4m3_encode(float(np.float32(x))))


def e4m3_value(b):
    return float(lib().uqo_e4m3_value(int(b)))


def prepare_query(q):
    """q [..., d] -> FP8 E4M3 bytes of the rotated query (Algorithm 1, Decode)."""
    q = _f32(q)
    d = _dim(q.shape[-1])
    out = np.empty(q.shape, np.uint8)
    lib().uqo_prepare_query_d(_ptr(q), q.size // d, _ptr(out), d)
    return out


def quantize_vector(x, c=C_DEFAULT, rotate=True):
    """One d-vector -> (codes[d] one per byte, scale_bytes[d / 32])."""
    x = _f32(x).reshape(-1)
    d = _dim(x.size)
    codes = np.empty(d, np.uint8)
    sb = np.empty(d // 32, np.uint8)
    lib().uqo_quantize_vector_d(_ptr(x), d, float(np.float32(c)), int(bool(rotate)), _ptr(codes), _ptr(sb))
    return codes, sb


def quantize_vectors(x, c=C_DEFAULT, rotate=True):
    """[..., d] -> (codes [..., d] one per byte, scale_bytes [..., d / 32])."""
    x = _f32(x)
    d = _dim(x.shape[-1])
    codes = np.empty(x.shape, np.uint8)
    sb = np.empty(x.shape[:-1] + (d // 32,), np.uint8)
    lib().uqo_quantize_vectors_d(_ptr(x), x.size // d, d, float(np.float32(c)), int(bool(rotate)), _ptr(codes),
                                 _ptr(sb))
    return codes, sb


def alloc_pools(num_pages, num_kv_heads, fill=0, head_dim=HEAD_DIM):
    """Codes pool (8 d bytes per page, head and K|V) and scales pool (d / 2)."""
    d = _dim(head_dim)
    codes = np.full(num_pages * num_kv_heads * 2 * 8 * d, fill, np.uint8)
    scales = np.full(num_pages * num_kv_heads * 2 * (d // 2), fill, np.uint8)
    return codes, scales


def quantize_kv(k, v, slot_mapping, num_pages, c=C_DEFAULT, rotate_v=True, pools=None):
    """k, v: [T, Hkv, 128] (any float dtype, converted exactly to fp32).

    Writes into ``pools`` (codes, scales) if given, else into zero-filled new
    pools, and returns them.
    """
    k = _f32(k)
    v = _f32(v)
    T, Hkv, D = k.shape
    D = _dim(D)
    assert v.shape == k.shape
    slots = np.ascontiguousarray(slot_mapping, dtype=np.int64)
    assert slots.shape == (T,)
    if pools is None:
        pools = alloc_pools(num_pages, Hkv, head_dim=D)
    codes, scales = pools
    assert codes.size == num_pages * Hkv * 16 * D
    lib().uqo_quantize_kv_d(_ptr(k), _ptr(v), T, Hkv, Hkv * D, _ptr(slots), int(num_pages), float(np.float32(c)),
                            int(bool(rotate_v)), _ptr(codes), _ptr(scales), D)
    return codes, scales


def load_vector(pools, num_kv_heads, page, head, kv, t, head_dim=HEAD_DIM):
    d = _dim(head_dim)
    codes = np.empty(d, np.uint8)
    sb = np.empty(d // 32, np.uint8)
    lib().uqo_load_vector_d(_ptr(pools[0]), _ptr(pools[1]), num_kv_heads, page, head, kv, t, _ptr(codes), _ptr(sb),
                            d)
    return codes, sb


def dequant_vector(pools, num_kv_heads, page, head, kv, t, head_dim=HEAD_DIM):
    d = _dim(head_dim)
    out = np.empty(d, np.float64)
    lib().uqo_dequant_vector_d(_ptr(pools[0]), _ptr(pools[1]), num_kv_heads, page, head, kv, t, _ptr(out), d)
    return out


def decode_attention(q, pools, page_table, context_lens, num_kv_heads, softmax_scale=None, rotate_v=True):
    """q [B, Hq, 128] -> fp64 attention output [B, Hq, 128] (Algorithm 1, Decode)."""
    q = _f32(q)
    B, Hq, D = q.shape
    D = _dim(D)
    assert Hq % num_kv_heads == 0
    pt = np.ascontiguousarray(page_table, dtype=np.int32)
    ctx = np.ascontiguousarray(context_lens, dtype=np.int32)
    assert pt.shape[0] == B and ctx.shape == (B,)
    if softmax_scale is None:
        softmax_scale = 1.0 / np.sqrt(D)
    out = np.empty((B, Hq, D), np.float64)
    lib().uqo_decode_attention_d(_ptr(q), B, Hq, num_kv_heads, _ptr(pools[0]), _ptr(pools[1]), _ptr(pt), pt.shape[1],
                                 _ptr(ctx), float(softmax_scale), int(bool(rotate_v)), _ptr(out), D)
    return out


def quantize_error(x, c_values, rotate=True, pow2=True):
    """Round-trip error of the FP4 encoder per constant c (section
    "Constant-Optimized Scaling"): rows x [..., 128] -> array [len(c), 2] of
    (sum of squared errors, sum of squares), fp64.  ``pow2`` selects the
    cache's scale 2^round(log2(c m)); otherwise the continuous s = c m."""
    x = _f32(x)
    assert x.shape[-1] == HEAD_DIM
    c = np.ascontiguousarray(np.atleast_1d(c_values), dtype=np.float32)
    sums = np.zeros((c.size, 2), np.float64)
    lib().uqo_quantize_error(_ptr(x), x.size // HEAD_DIM, int(bool(rotate)), int(bool(pow2)), c.size, _ptr(c),
                             _ptr(sums))
    return sums


# ---------------------------------------------------------------------------
# Ultra-TQ comparison cache (appendix "Calibrated LUT int4 KV Encoding
# (Ultra-TQ)"); readings T1-T5 in uq_oracle.c.

TQ_BLOCK = 2368


def _levels(levels):
    lv = np.ascontiguousarray(levels, dtype=np.float32)
    assert lv.shape == (16,)
    return lv


def bf16_rne(x):
    return float(lib().uqo_bf16_rne(float(np.float32(x))))


def tq4_norm(x):
    """Reading T2: the l2 norm of the fp32 vector x [128], rounded once to fp32."""
    x = _f32(x).reshape(HEAD_DIM)
    return float(lib().uqo_tq4_norm(_ptr(x)))


def tq4_index(x, n, levels):
    """Reading T3: index of the BF16 level nearest to x / n (ties to the lower)."""
    return int(lib().uqo_tq4_index(float(np.float32(x)), float(np.float32(n)), _ptr(_levels(levels))))


def tq4_encode_vector(k, v, levels):
    """One token -> (K indices [128], norm, V codes [128], s [4], z [4])."""
    k = _f32(k).reshape(HEAD_DIM)
    v = _f32(v).reshape(HEAD_DIM)
    kidx = np.empty(HEAD_DIM, np.uint8)
    vcode = np.empty(HEAD_DIM, np.uint8)
    n = np.empty(1, np.float32)
    s = np.empty(4, np.float32)
    z = np.empty(4, np.float32)
    lib().uqo_tq4_encode_vector(_ptr(k), _ptr(v), _ptr(_levels(levels)), _ptr(kidx), _ptr(n), _ptr(vcode), _ptr(s),
                                _ptr(z))
    return kidx, float(n[0]), vcode, s, z


def tq4_alloc_cache(num_pages, num_kv_heads, fill=0):
    return np.full(num_pages * num_kv_heads * TQ_BLOCK, fill, np.uint8)


def tq4_write(k, v, slot_mapping, num_pages, levels, cache=None):
    """k, v: [T, Hkv, 128] -> the Ultra-TQ cache (written into ``cache``)."""
    k = _f32(k)
    v = _f32(v)
    T, Hkv, D = k.shape
    assert D == HEAD_DIM and v.shape == k.shape
    slots = np.ascontiguousarray(slot_mapping, dtype=np.int64)
    if cache is None:
        cache = tq4_alloc_cache(num_pages, Hkv)
    lib().uqo_tq4_write(_ptr(k), _ptr(v), T, Hkv, Hkv * HEAD_DIM, _ptr(slots), int(num_pages), _ptr(_levels(levels)),
                        _ptr(cache))
    return cache


def tq4_load(cache, num_kv_heads, page, head, t):
    kidx = np.empty(HEAD_DIM, np.uint8)
    vcode = np.empty(HEAD_DIM, np.uint8)
    n = np.empty(1, np.float32)
    s = np.empty(4, np.float32)
    z = np.empty(4, np.float32)
    lib().uqo_tq4_load(_ptr(cache), num_kv_heads, page, head, t, _ptr(kidx), _ptr(n), _ptr(vcode), _ptr(s), _ptr(z))
    return kidx, float(n[0]), vcode, s, z


def tq4_dequant(cache, num_kv_heads, page, head, t, levels):
    """(rotated K, V) of one token as fp64 [128] each."""
    kv = np.empty(HEAD_DIM, np.float64)
    vv = np.empty(HEAD_DIM, np.float64)
    lib().uqo_tq4_dequant(_ptr(cache), num_kv_heads, page, head, t, _ptr(_levels(levels)), _ptr(kv), _ptr(vv))
    return kv, vv


def tq4_decode_attention(q, cache, page_table, context_lens, num_kv_heads, levels, softmax_scale=None):
    """q [B, Hq, 128] -> fp64 attention over the Ultra-TQ cache."""
    q = _f32(q)
    B, Hq, D = q.shape
    assert D == HEAD_DIM and Hq % num_kv_heads == 0
    pt = np.ascontiguousarray(page_table, dtype=np.int32)
    ctx = np.ascontiguousarray(context_lens, dtype=np.int32)
    if softmax_scale is None:
        softmax_scale = 1.0 / np.sqrt(HEAD_DIM)
    out = np.empty((B, Hq, HEAD_DIM), np.float64)
    lib().uqo_tq4_decode_attention(_ptr(q), B, Hq, num_kv_heads, _ptr(cache), _ptr(pt), pt.shape[1], _ptr(ctx),
                                   float(softmax_scale), _ptr(_levels(levels)), _ptr(out))
    return out
