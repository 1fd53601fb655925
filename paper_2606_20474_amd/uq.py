"""Python binding of libuq (``include/uq.h``): argument marshalling only.

Every step of the path runs in the HIP kernels of ``libuq.so``; this module
turns torch tensors into device pointers and the current torch stream into a
``hipStream_t``, calls the C entry point of the same name and raises
:class:`UQError` on a non-OK status.  There is no fallback: if the library is
missing, importing this module fails.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
# UQ_LIB names another build of the same sources (the CPU sanitizer test
# loads a host-sanitised build that way, in a subprocess of its own)
LIB_PATH = os.environ.get("UQ_LIB") or os.path.join(_PKG, "libuq.so")

UQ_OK, UQ_ERR_INVALID_ARGUMENT, UQ_ERR_UNSUPPORTED, UQ_ERR_WORKSPACE_TOO_SMALL, UQ_ERR_HIP = range(5)
UQ_F32, UQ_BF16, UQ_F16, UQ_FP8_E4M3 = range(4)
NOALLOC_SCRATCH_BYTES = 32 << 20   # UQ_NOALLOC_SCRATCH_BYTES
PROBE_STREAM_BLOCKS = 2048         # UQ_PROBE_STREAM_BLOCKS
PROBE_MFMA_FP4_FP8, PROBE_MFMA_FP8_FP8, PROBE_MFMA_BF16, PROBE_MFMA_FP8_FP4 = range(4)

HEAD_DIM = 128
PAGE_SIZE = 16
GROUP_SIZE = 32
TILE_CODES = 1024
TILE_SCALES = 64

# Every symbol include/uq.h declares.
EXPORTS = (
    "uq_status_string", "uq_version", "uq_quantize_kv", "uq_prepare_query", "uq_decode_workspace_bytes",
    "uq_default_partition", "uq_decode_attention", "uq_decode_partials", "uq_decode_merge", "uq_decode_step",
    "uq_decode_step_partials", "uq_ref_cache_bytes", "uq_ref_write_kv", "uq_ref_decode_workspace_bytes",
    "uq_ref_decode_attention", "uq_ref_decode_partials", "uq_ref_decode_merge", "uq_ref_decode_step",
    "uq_ref_decode_step_partials", "uq_decode_cascade_workspace_bytes", "uq_decode_cascade",
    "uq_decode_cascade_partials", "uq_decode_cascade_merge", "uq_ref_decode_cascade",
    "uq_ref_decode_cascade_partials", "uq_ref_decode_cascade_merge", "uq_quantize_error", "uq_time_next_launch",
    "uq_decode_attention_noalloc", "uq_decode_attention_scaled_pv", "uq_probe_stream_read", "uq_probe_page_gather",
    "uq_probe_page_gather_cascade", "uq_probe_mfma",
)

UQ_REF_FP8_E4M3, UQ_REF_BF16, UQ_REF_TQ4 = 1, 2, 3


class UQError(RuntimeError):
    def __init__(self, status: int, call: str):
        self.status = status
        super().__init__(f"{call} failed: {status_string(status)}")


class uq_cache_desc(ctypes.Structure):
    _fields_ = [
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("group_size", ctypes.c_int32),
        ("num_pages", ctypes.c_int64),
        ("c", ctypes.c_float),
        ("rotate_v", ctypes.c_int32),
    ]


class uq_ref_cache_desc(ctypes.Structure):
    _fields_ = [
        ("num_kv_heads", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("page_size", ctypes.c_int32),
        ("format", ctypes.c_int32),
        ("num_pages", ctypes.c_int64),
        ("k_scale", ctypes.c_float),
        ("v_scale", ctypes.c_float),
        ("codebook", ctypes.c_void_p),
    ]


class uq_shared_prefix(ctypes.Structure):
    _fields_ = [
        ("pages", ctypes.c_void_p),
        ("lens", ctypes.c_void_p),
        ("num_tokens", ctypes.c_int32),
        ("partition_tokens", ctypes.c_int32),
    ]


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run `python -m paper_2606_20474_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    vp, i32, i64, f32, sz = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_size_t
    D = ctypes.POINTER(uq_cache_desc)
    L.uq_status_string.argtypes = [i32]
    L.uq_status_string.restype = ctypes.c_char_p
    L.uq_version.restype = i32
    L.uq_quantize_kv.argtypes = [D, vp, vp, i32, i64, i64, vp, i32, i32, vp, vp, vp, vp]
    L.uq_quantize_kv.restype = i32
    L.uq_prepare_query.argtypes = [D, vp, i32, i64, vp, vp]
    L.uq_prepare_query.restype = i32
    L.uq_quantize_error.argtypes = [vp, i32, i64, i64, i32, i32, i32, vp, vp, vp]
    L.uq_quantize_error.restype = i32
    L.uq_time_next_launch.argtypes = [vp, vp]
    L.uq_time_next_launch.restype = i32
    L.uq_decode_workspace_bytes.argtypes = [D, i32, i32, i32, i32]
    L.uq_decode_workspace_bytes.restype = sz
    L.uq_default_partition.argtypes = [D, i32, i32, i32]
    L.uq_default_partition.restype = i32
    L.uq_decode_attention.argtypes = [D, vp, i32, i32, i32, vp, vp, vp, i32, vp, i32, f32, i32, vp, sz, vp, i32, vp]
    L.uq_decode_attention.restype = i32
    L.uq_decode_partials.argtypes = [D, vp, i32, i32, i32, vp, vp, vp, i32, vp, i32, f32, i32, vp, sz, vp, i32, vp]
    L.uq_decode_partials.restype = i32
    L.uq_decode_merge.argtypes = [D, i32, i32, vp, i32, i32, vp, sz, vp, i32, vp]
    L.uq_decode_merge.restype = i32
    L.uq_decode_attention_scaled_pv.argtypes = [D, vp, i32, i32, i32, vp, vp, vp, i32, vp, i32, f32, i32, vp, sz, vp,
                                                i32, vp]
    L.uq_decode_attention_scaled_pv.restype = i32
    L.uq_decode_attention_noalloc.argtypes = [D, vp, i32, i32, i32, vp, vp, vp, i32, vp, i32, f32, i32, vp, i32, vp]
    L.uq_decode_attention_noalloc.restype = i32
    L.uq_probe_stream_read.argtypes = [vp, sz, vp, vp]
    L.uq_probe_stream_read.restype = i32
    L.uq_probe_page_gather.argtypes = [D, i32, i32, vp, vp, vp, i32, vp, i32, i32, vp, sz, vp]
    L.uq_probe_page_gather.restype = i32
    L.uq_probe_page_gather_cascade.argtypes = [D, i32, i32, vp, vp, vp, i32, vp, i32, vp, i32, vp, sz, vp, sz, vp]
    L.uq_probe_page_gather_cascade.restype = i32
    L.uq_probe_mfma.argtypes = [i32, vp, vp, vp, vp, i32, vp, vp]
    L.uq_probe_mfma.restype = i32
    for name in ("uq_decode_step", "uq_decode_step_partials"):
        fn = getattr(L, name)
        fn.argtypes = [D, vp, i32, vp, vp, i32, i32, i32, vp, vp, vp, i32, vp, i32, f32, i32, vp, sz, vp, i32, vp]
        fn.restype = i32
    R = ctypes.POINTER(uq_ref_cache_desc)
    S = ctypes.POINTER(uq_shared_prefix)
    L.uq_decode_cascade_workspace_bytes.argtypes = [i32, i32, i32, i32, i32, S]
    L.uq_decode_cascade_workspace_bytes.restype = sz
    for name in ("uq_decode_cascade", "uq_decode_cascade_partials"):
        fn = getattr(L, name)
        fn.argtypes = [D, vp, i32, vp, vp, i32, i32, i32, vp, vp, vp, i32, vp, i32, S, f32, i32, vp, sz, vp, i32, vp]
        fn.restype = i32
    L.uq_decode_cascade_merge.argtypes = [D, i32, i32, vp, i32, S, i32, vp, sz, vp, i32, vp]
    L.uq_decode_cascade_merge.restype = i32
    for name in ("uq_ref_decode_cascade", "uq_ref_decode_cascade_partials"):
        fn = getattr(L, name)
        fn.argtypes = [R, vp, i32, vp, vp, i32, i32, i32, vp, vp, i32, vp, i32, S, f32, i32, vp, sz, vp, i32, vp]
        fn.restype = i32
    L.uq_ref_decode_cascade_merge.argtypes = [R, i32, i32, vp, i32, S, i32, vp, sz, vp, i32, vp]
    L.uq_ref_decode_cascade_merge.restype = i32
    L.uq_ref_cache_bytes.argtypes = [R]
    L.uq_ref_cache_bytes.restype = sz
    L.uq_ref_write_kv.argtypes = [R, vp, vp, i32, i64, i64, vp, i32, i32, vp, vp, vp]
    L.uq_ref_write_kv.restype = i32
    L.uq_ref_decode_workspace_bytes.argtypes = [R, i32, i32, i32, i32]
    L.uq_ref_decode_workspace_bytes.restype = sz
    for name in ("uq_ref_decode_attention", "uq_ref_decode_partials"):
        fn = getattr(L, name)
        fn.argtypes = [R, vp, i32, i32, i32, vp, vp, i32, vp, i32, f32, i32, vp, sz, vp, i32, vp]
        fn.restype = i32
    L.uq_ref_decode_merge.argtypes = [R, i32, i32, vp, i32, i32, vp, sz, vp, i32, vp]
    L.uq_ref_decode_merge.restype = i32
    for name in ("uq_ref_decode_step", "uq_ref_decode_step_partials"):
        fn = getattr(L, name)
        fn.argtypes = [R, vp, i32, vp, vp, i32, i32, i32, vp, vp, i32, vp, i32, f32, i32, vp, sz, vp, i32, vp]
        fn.restype = i32
    return L


lib = _load()


def status_string(status: int) -> str:
    return lib.uq_status_string(int(status)).decode()


def _check(status: int, call: str):
    if status != UQ_OK:
        raise UQError(status, call)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


_ROWS = (torch.float32, torch.bfloat16, torch.float16)               # K/V and query rows
_QUERY = _ROWS + (torch.uint8, torch.float8_e4m3fn)                    # ... or a pre-cast FP8 query
_OUT = (torch.float32, torch.bfloat16)
_I32 = (torch.int32,)
_U8 = (torch.uint8,)


def _need(t, name, dtypes, shape=None, min_numel=None, contiguous=True):
    """The checks the C ABI cannot make, since it sees raw pointers only: a
    HIP tensor on the current device, of one of `dtypes`, contiguous (unless
    the caller checks strides itself), of `shape` (None matches any size)
    and with at least `min_numel` elements.  Raises before anything is
    enqueued."""
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name}: a torch.Tensor expected, got {type(t).__name__}")
    if not t.is_cuda:
        raise ValueError(f"{name}: a tensor on the GPU expected, got one on {t.device}")
    if t.device.index != torch.cuda.current_device():
        raise ValueError(f"{name}: on {t.device}, but the current device is cuda:{torch.cuda.current_device()}")
    if t.dtype not in dtypes:
        raise TypeError(f"{name}: dtype {t.dtype}, expected one of {[str(d) for d in dtypes]}")
    if contiguous and not t.is_contiguous():
        raise ValueError(f"{name}: a contiguous tensor expected")
    if shape is not None and (t.dim() != len(shape) or any(w is not None and w != n for w, n in zip(shape, t.shape))):
        raise ValueError(f"{name}: shape {tuple(t.shape)}, expected {tuple('*' if w is None else w for w in shape)}")
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError(f"{name}: {t.numel()} elements, at least {min_numel} needed")
    return t


def _rows(k, v, num_kv_heads, head_dim, token_stride):
    """K and V rows [T, Hkv, head_dim]: channels and heads contiguous, one
    token stride for both; returns the token stride in elements."""
    for t, name in ((k, "k"), (v, "v")):
        _need(t, name, _ROWS, (None, num_kv_heads, head_dim), contiguous=False)
        if t.stride(2) != 1 or t.stride(1) != head_dim:
            raise ValueError(f"{name}: heads and channels of a token must be contiguous")
    if v.shape[0] != k.shape[0] or v.dtype != k.dtype:
        raise ValueError("k and v: the same number of tokens and dtype expected")
    if token_stride is None:
        token_stride = k.stride(0)
    if k.shape[0] > 1 and (k.stride(0) != token_stride or v.stride(0) != token_stride):
        raise ValueError(f"k and v: token stride {token_stride} expected, got {k.stride(0)} and {v.stride(0)}")
    return token_stride


def _table(page_table, context_lens, B):
    """Page table int32 [>= B, max_pages_per_seq] and context lengths int32 [B]."""
    _need(page_table, "page_table", _I32, (None, None))
    if page_table.shape[0] < B:
        raise ValueError(f"page_table: {page_table.shape[0]} rows for a batch of {B}")
    _need(context_lens, "context_lens", _I32, (B,))


def _write_table(page_table, max_pages_per_seq):
    """Page table of a write (int32 [num_seqs, width]) and the row length
    the kernel indexes it with: 0 selects the width; an explicit value must
    lie in 1..width, since the kernel reads page_table[seq * mpps + page]
    and a longer row would read past the tensor.  Returns (num_seqs, mpps),
    (0, 0) without a table."""
    if page_table is None:
        return 0, 0
    if isinstance(page_table, torch.Tensor) and page_table.dim() == 2:
        width = page_table.shape[1]
        mpps = max_pages_per_seq or width
        if not 1 <= mpps <= width:
            raise ValueError(f"max_pages_per_seq: {mpps}, expected 1..{width} (the page table's row length)")
    _need(page_table, "page_table", _I32, (None, None))
    return page_table.shape[0], max_pages_per_seq or page_table.shape[1]


def _q_out(q, out, head_dim):
    _need(q, "q", _QUERY, (None, None, head_dim))
    B, Hq = q.shape[0], q.shape[1]
    if out is not None:
        _need(out, "out", _OUT, (B, Hq, head_dim))
    return B, Hq


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


_DT = {torch.float32: UQ_F32, torch.bfloat16: UQ_BF16, torch.float16: UQ_F16, torch.uint8: UQ_FP8_E4M3,
       torch.float8_e4m3fn: UQ_FP8_E4M3}


@dataclass
class CacheDesc:
    """Python mirror of ``uq_cache_desc`` (head_dim 64, 128 or 256; the step,
    cascade and FP8-query calls take 128 only)."""
    num_kv_heads: int
    num_pages: int
    c: float = 0.156
    rotate_v: bool = True
    head_dim: int = HEAD_DIM
    page_size: int = PAGE_SIZE
    group_size: int = GROUP_SIZE

    def c_struct(self):
        return uq_cache_desc(self.num_kv_heads, self.head_dim, self.page_size, self.group_size, self.num_pages,
                             self.c, int(bool(self.rotate_v)))

    def codes_bytes(self):
        return self.num_pages * self.num_kv_heads * 2 * 8 * self.head_dim

    def scales_bytes(self):
        return self.num_pages * self.num_kv_heads * 2 * (self.head_dim // 2)

    def alloc_pools(self, device="cuda", fill=None):
        codes = torch.empty(self.codes_bytes(), dtype=torch.uint8, device=device)
        scales = torch.empty(self.scales_bytes(), dtype=torch.uint8, device=device)
        if fill is not None:
            codes.fill_(fill)
            scales.fill_(fill)
        return codes, scales


def _pools(desc: CacheDesc, codes, scales):
    _need(codes, "codes", _U8, min_numel=desc.codes_bytes())
    _need(scales, "scales", _U8, min_numel=desc.scales_bytes())


def quantize_kv(desc: CacheDesc, k, v, slot_mapping, codes, scales, page_table=None, max_pages_per_seq=0,
                token_stride=None, stream=None):
    """k, v: [T, Hkv, head_dim] (or strided rows); slot_mapping int64 [T]."""
    num_seqs, mpps = _write_table(page_table, max_pages_per_seq)
    token_stride = _rows(k, v, desc.num_kv_heads, desc.head_dim, token_stride)
    T = k.shape[0]
    _need(slot_mapping, "slot_mapping", (torch.int64,), (T,))
    _pools(desc, codes, scales)
    d = desc.c_struct()
    st = lib.uq_quantize_kv(ctypes.byref(d), _ptr(k), _ptr(v), _DT[k.dtype], T, token_stride, _ptr(page_table),
                            num_seqs, mpps, _ptr(slot_mapping), _ptr(codes), _ptr(scales), _stream(stream))
    _check(st, "uq_quantize_kv")


def prepare_query(desc: CacheDesc, q, out=None, stream=None):
    _need(q, "q", _ROWS)
    if q.numel() % HEAD_DIM:
        raise ValueError(f"q: rows of {HEAD_DIM} channels expected")
    rows = q.numel() // HEAD_DIM
    if out is None:
        out = torch.empty(q.shape, dtype=torch.uint8, device=q.device)
    _need(out, "out", (torch.uint8, torch.float8_e4m3fn), min_numel=q.numel())
    d = desc.c_struct()
    _check(lib.uq_prepare_query(ctypes.byref(d), _ptr(q), _DT[q.dtype], rows, _ptr(out), _stream(stream)),
           "uq_prepare_query")
    return out


def time_next_launch(start, stop):
    """The next decode partition or quantize-on-write launch of this thread
    sets the torch CUDA events `start` and `stop` to its kernel's own start
    and end (record them once beforehand, so that their HIP events exist);
    None, None clears."""
    if start is None and stop is None:
        _check(lib.uq_time_next_launch(None, None), "uq_time_next_launch")
        return
    if not start.cuda_event or not stop.cuda_event:
        raise ValueError("record the events once before passing them")
    _check(lib.uq_time_next_launch(ctypes.c_void_p(start.cuda_event), ctypes.c_void_p(stop.cuda_event)),
           "uq_time_next_launch")


def quantize_error(x, c_values, rotate=True, pow2=True, sums=None, stream=None):
    """Round-trip error of the encoder per constant c: x rows [N, 128]
    (last dimension contiguous), c_values float32 [n] on the device ->
    ``sums`` float64 [n, 2] (sum of squared errors, sum of squares),
    accumulated into ``sums`` if given, else into a new zeroed tensor."""
    _need(x, "x", _ROWS, contiguous=False)
    rows = x.reshape(-1, HEAD_DIM) if x.dim() != 2 else x
    if rows.shape[-1] != HEAD_DIM or rows.stride(-1) != 1:
        raise ValueError("rows of 128 contiguous channels expected")
    c = c_values.to(device=x.device, dtype=torch.float32).contiguous()
    if sums is None:
        sums = torch.zeros((c.numel(), 2), dtype=torch.float64, device=x.device)
    _need(sums, "sums", (torch.float64,), (c.numel(), 2))
    st = lib.uq_quantize_error(_ptr(rows), _DT[x.dtype], rows.shape[0], rows.stride(0), int(bool(rotate)),
                               int(bool(pow2)), c.numel(), _ptr(c), _ptr(sums), _stream(stream))
    _check(st, "uq_quantize_error")
    return sums


def workspace_bytes(desc: CacheDesc, batch, num_q_heads, max_context, partition_tokens=0):
    d = desc.c_struct()
    return int(lib.uq_decode_workspace_bytes(ctypes.byref(d), batch, num_q_heads, max_context, partition_tokens))


def default_partition(desc: CacheDesc, batch, num_q_heads, max_context):
    d = desc.c_struct()
    return int(lib.uq_default_partition(ctypes.byref(d), batch, num_q_heads, max_context))


def alloc_workspace(desc: CacheDesc, batch, num_q_heads, max_context, partition_tokens=0, device="cuda"):
    n = workspace_bytes(desc, batch, num_q_heads, max_context, partition_tokens)
    return torch.empty(n, dtype=torch.uint8, device=device)


def decode_attention(desc: CacheDesc, q, codes, scales, page_table, context_lens, max_context, softmax_scale=None,
                     partition_tokens=0, workspace=None, out=None, out_dtype=torch.float32, q_dtype=None,
                     stream=None):
    """q: [B, Hq, head_dim] -> out [B, Hq, head_dim]."""
    B, Hq = _q_out(q, out, desc.head_dim)
    _pools(desc, codes, scales)
    _table(page_table, context_lens, B)
    if softmax_scale is None:
        softmax_scale = desc.head_dim ** -0.5
    if workspace is None:
        workspace = alloc_workspace(desc, B, Hq, max_context, partition_tokens, q.device)
    _need(workspace, "workspace", _U8)
    if out is None:
        out = torch.empty((B, Hq, desc.head_dim), dtype=out_dtype, device=q.device)
    d = desc.c_struct()
    qdt = _DT[q.dtype] if q_dtype is None else q_dtype
    st = lib.uq_decode_attention(ctypes.byref(d), _ptr(q), qdt, B, Hq, _ptr(codes), _ptr(scales), _ptr(page_table),
                                 page_table.shape[1], _ptr(context_lens), max_context, softmax_scale,
                                 partition_tokens, _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype],
                                 _stream(stream))
    _check(st, "uq_decode_attention")
    return out


def decode_attention_scaled_pv(desc: CacheDesc, q, codes, scales, page_table, context_lens, max_context,
                               softmax_scale=None, partition_tokens=0, workspace=None, out=None,
                               out_dtype=torch.float32, q_dtype=None, stream=None):
    """decode_attention with PV on the block-scaled matrix instruction (the
    prototype of include/uq.h; head size 128)."""
    B, Hq = _q_out(q, out, desc.head_dim)
    _pools(desc, codes, scales)
    _table(page_table, context_lens, B)
    if softmax_scale is None:
        softmax_scale = desc.head_dim ** -0.5
    if workspace is None:
        workspace = alloc_workspace(desc, B, Hq, max_context, partition_tokens, q.device)
    _need(workspace, "workspace", _U8)
    if out is None:
        out = torch.empty((B, Hq, desc.head_dim), dtype=out_dtype, device=q.device)
    d = desc.c_struct()
    qdt = _DT[q.dtype] if q_dtype is None else q_dtype
    st = lib.uq_decode_attention_scaled_pv(ctypes.byref(d), _ptr(q), qdt, B, Hq, _ptr(codes), _ptr(scales),
                                           _ptr(page_table), page_table.shape[1], _ptr(context_lens), max_context,
                                           softmax_scale, partition_tokens, _ptr(workspace), workspace.numel(),
                                           _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_decode_attention_scaled_pv")
    return out


def decode_attention_noalloc(desc: CacheDesc, q, codes, scales, page_table, context_lens, max_context, out,
                             softmax_scale=None, partition_tokens=0, q_dtype=None, stream=None):
    """decode_attention with its partials in the library's own device array
    (no workspace, nothing allocated by the call); ``out`` [B, Hq, head_dim]
    is the caller's."""
    B, Hq = _q_out(q, out, desc.head_dim)
    _pools(desc, codes, scales)
    _table(page_table, context_lens, B)
    if softmax_scale is None:
        softmax_scale = desc.head_dim ** -0.5
    d = desc.c_struct()
    qdt = _DT[q.dtype] if q_dtype is None else q_dtype
    st = lib.uq_decode_attention_noalloc(ctypes.byref(d), _ptr(q), qdt, B, Hq, _ptr(codes), _ptr(scales),
                                         _ptr(page_table), page_table.shape[1], _ptr(context_lens), max_context,
                                         softmax_scale, partition_tokens, _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_decode_attention_noalloc")
    return out


def decode_partials(desc: CacheDesc, q, codes, scales, page_table, context_lens, max_context, softmax_scale,
                    partition_tokens, workspace, out, q_dtype=None, stream=None):
    """First launch of decode_attention (partition kernel)."""
    B, Hq = _q_out(q, out, desc.head_dim)
    _pools(desc, codes, scales)
    _table(page_table, context_lens, B)
    _need(workspace, "workspace", _U8)
    d = desc.c_struct()
    qdt = _DT[q.dtype] if q_dtype is None else q_dtype
    st = lib.uq_decode_partials(ctypes.byref(d), _ptr(q), qdt, B, Hq, _ptr(codes), _ptr(scales), _ptr(page_table),
                                page_table.shape[1], _ptr(context_lens), max_context, softmax_scale, partition_tokens,
                                _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_decode_partials")
    return out


def _new_token(k_new, v_new, B, num_kv_heads):
    """The decode step's new tokens: [B, Hkv, 128] each, contiguous, one dtype."""
    _need(k_new, "k_new", _ROWS, (B, num_kv_heads, HEAD_DIM))
    _need(v_new, "v_new", (k_new.dtype,), (B, num_kv_heads, HEAD_DIM))


def decode_step(desc: CacheDesc, q, k_new, v_new, codes, scales, page_table, context_lens, max_context,
                softmax_scale=None, partition_tokens=0, workspace=None, out=None, out_dtype=torch.float32,
                q_dtype=None, stream=None, partials_only=False):
    """Write each sequence's new token (k_new, v_new: [B, Hkv, 128]) at its
    last position, then decode attention; q: [B, Hq, 128] -> out."""
    B, Hq = _q_out(q, out, desc.head_dim)
    _pools(desc, codes, scales)
    _table(page_table, context_lens, B)
    _new_token(k_new, v_new, B, desc.num_kv_heads)
    if softmax_scale is None:
        softmax_scale = desc.head_dim ** -0.5
    if workspace is None:
        workspace = alloc_workspace(desc, B, Hq, max_context, partition_tokens, q.device)
    _need(workspace, "workspace", _U8)
    if out is None:
        out = torch.empty((B, Hq, desc.head_dim), dtype=out_dtype, device=q.device)
    d = desc.c_struct()
    qdt = _DT[q.dtype] if q_dtype is None else q_dtype
    fn = lib.uq_decode_step_partials if partials_only else lib.uq_decode_step
    st = fn(ctypes.byref(d), _ptr(q), qdt, _ptr(k_new), _ptr(v_new), _DT[k_new.dtype], B, Hq, _ptr(codes),
            _ptr(scales), _ptr(page_table), page_table.shape[1], _ptr(context_lens), max_context, softmax_scale,
            partition_tokens, _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_decode_step_partials" if partials_only else "uq_decode_step")
    return out


def decode_merge(desc: CacheDesc, batch, num_q_heads, context_lens, max_context, partition_tokens, workspace, out,
                 stream=None):
    """Second launch of decode_attention (merge of the partitions)."""
    _need(context_lens, "context_lens", _I32, (batch,))
    _need(workspace, "workspace", _U8)
    _need(out, "out", _OUT, (batch, num_q_heads, desc.head_dim))
    d = desc.c_struct()
    st = lib.uq_decode_merge(ctypes.byref(d), batch, num_q_heads, _ptr(context_lens), max_context, partition_tokens,
                             _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_decode_merge")
    return out


# ---------------------------------------------------------------------------
# Plain comparison caches (FP8 E4M3 with per-tensor scales, BF16)


@dataclass
class RefCacheDesc:
    """Python mirror of ``uq_ref_cache_desc``; ``fmt`` is "fp8", "bf16" or
    "tq4" (the Ultra-TQ codebook cache; ``codebook``: 16 ascending levels,
    default the theoretical codebook for head size 128)."""
    num_kv_heads: int
    num_pages: int
    fmt: str = "fp8"
    k_scale: float = 1.0
    v_scale: float = 1.0
    head_dim: int = HEAD_DIM
    page_size: int = PAGE_SIZE
    codebook: object = None

    def __post_init__(self):
        if self.fmt == "tq4" and self.codebook is None:
            from .codebook import default_tq_codebook
            self.codebook = default_tq_codebook(self.head_dim)
        if self.codebook is not None:
            import numpy as np
            self.codebook = np.ascontiguousarray(self.codebook, dtype=np.float32)

    def c_struct(self):
        code = {"fp8": UQ_REF_FP8_E4M3, "bf16": UQ_REF_BF16, "tq4": UQ_REF_TQ4}.get(self.fmt, 0)
        cb = None if self.codebook is None else ctypes.c_void_p(self.codebook.ctypes.data)
        return uq_ref_cache_desc(self.num_kv_heads, self.head_dim, self.page_size, code, self.num_pages,
                                 self.k_scale, self.v_scale, cb)

    def cache_bytes(self):
        d = self.c_struct()
        return int(lib.uq_ref_cache_bytes(ctypes.byref(d)))

    def alloc_cache(self, device="cuda", fill=None):
        n = self.cache_bytes()
        if n == 0:
            raise UQError(UQ_ERR_INVALID_ARGUMENT, "uq_ref_cache_bytes")
        cache = torch.empty(n, dtype=torch.uint8, device=device)
        if fill is not None:
            cache.fill_(fill)
        return cache


def _cache(desc: RefCacheDesc, cache):
    _need(cache, "cache", _U8, min_numel=desc.cache_bytes())


def ref_write_kv(desc: RefCacheDesc, k, v, slot_mapping, cache, page_table=None, max_pages_per_seq=0,
                 token_stride=None, stream=None):
    num_seqs, mpps = _write_table(page_table, max_pages_per_seq)
    token_stride = _rows(k, v, desc.num_kv_heads, desc.head_dim, token_stride)
    T = k.shape[0]
    _need(slot_mapping, "slot_mapping", (torch.int64,), (T,))
    _cache(desc, cache)
    d = desc.c_struct()
    st = lib.uq_ref_write_kv(ctypes.byref(d), _ptr(k), _ptr(v), _DT[k.dtype], T, token_stride, _ptr(page_table),
                             num_seqs, mpps, _ptr(slot_mapping), _ptr(cache), _stream(stream))
    _check(st, "uq_ref_write_kv")


def ref_workspace_bytes(desc: RefCacheDesc, batch, num_q_heads, max_context, partition_tokens=0):
    d = desc.c_struct()
    return int(lib.uq_ref_decode_workspace_bytes(ctypes.byref(d), batch, num_q_heads, max_context, partition_tokens))


def ref_alloc_workspace(desc: RefCacheDesc, batch, num_q_heads, max_context, partition_tokens=0, device="cuda"):
    n = ref_workspace_bytes(desc, batch, num_q_heads, max_context, partition_tokens)
    return torch.empty(n, dtype=torch.uint8, device=device)


def ref_decode_attention(desc: RefCacheDesc, q, cache, page_table, context_lens, max_context, softmax_scale=None,
                         partition_tokens=0, workspace=None, out=None, out_dtype=torch.float32, stream=None):
    B, Hq = _q_out(q, out, HEAD_DIM)
    _cache(desc, cache)
    _table(page_table, context_lens, B)
    if softmax_scale is None:
        softmax_scale = HEAD_DIM ** -0.5
    if workspace is None:
        workspace = ref_alloc_workspace(desc, B, Hq, max_context, partition_tokens, q.device)
    _need(workspace, "workspace", _U8)
    if out is None:
        out = torch.empty((B, Hq, HEAD_DIM), dtype=out_dtype, device=q.device)
    d = desc.c_struct()
    st = lib.uq_ref_decode_attention(ctypes.byref(d), _ptr(q), _DT[q.dtype], B, Hq, _ptr(cache), _ptr(page_table),
                                     page_table.shape[1], _ptr(context_lens), max_context, softmax_scale,
                                     partition_tokens, _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype],
                                     _stream(stream))
    _check(st, "uq_ref_decode_attention")
    return out


def ref_decode_partials(desc: RefCacheDesc, q, cache, page_table, context_lens, max_context, softmax_scale,
                        partition_tokens, workspace, out, stream=None):
    B, Hq = _q_out(q, out, HEAD_DIM)
    _cache(desc, cache)
    _table(page_table, context_lens, B)
    _need(workspace, "workspace", _U8)
    d = desc.c_struct()
    st = lib.uq_ref_decode_partials(ctypes.byref(d), _ptr(q), _DT[q.dtype], B, Hq, _ptr(cache), _ptr(page_table),
                                    page_table.shape[1], _ptr(context_lens), max_context, softmax_scale,
                                    partition_tokens, _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype],
                                    _stream(stream))
    _check(st, "uq_ref_decode_partials")
    return out


def ref_decode_merge(desc: RefCacheDesc, batch, num_q_heads, context_lens, max_context, partition_tokens, workspace,
                     out, stream=None):
    _need(context_lens, "context_lens", _I32, (batch,))
    _need(workspace, "workspace", _U8)
    _need(out, "out", _OUT, (batch, num_q_heads, HEAD_DIM))
    d = desc.c_struct()
    st = lib.uq_ref_decode_merge(ctypes.byref(d), batch, num_q_heads, _ptr(context_lens), max_context,
                                 partition_tokens, _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype],
                                 _stream(stream))
    _check(st, "uq_ref_decode_merge")
    return out


def ref_decode_step(desc: RefCacheDesc, q, k_new, v_new, cache, page_table, context_lens, max_context,
                    softmax_scale=None, partition_tokens=0, workspace=None, out=None, out_dtype=torch.float32,
                    stream=None, partials_only=False):
    B, Hq = _q_out(q, out, HEAD_DIM)
    _cache(desc, cache)
    _table(page_table, context_lens, B)
    _new_token(k_new, v_new, B, desc.num_kv_heads)
    if softmax_scale is None:
        softmax_scale = HEAD_DIM ** -0.5
    if workspace is None:
        workspace = ref_alloc_workspace(desc, B, Hq, max_context, partition_tokens, q.device)
    _need(workspace, "workspace", _U8)
    if out is None:
        out = torch.empty((B, Hq, HEAD_DIM), dtype=out_dtype, device=q.device)
    d = desc.c_struct()
    fn = lib.uq_ref_decode_step_partials if partials_only else lib.uq_ref_decode_step
    st = fn(ctypes.byref(d), _ptr(q), _DT[q.dtype], _ptr(k_new), _ptr(v_new), _DT[k_new.dtype], B, Hq, _ptr(cache),
            _ptr(page_table), page_table.shape[1], _ptr(context_lens), max_context, softmax_scale, partition_tokens,
            _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_ref_decode_step_partials" if partials_only else "uq_ref_decode_step")
    return out


# ---------------------------------------------------------------------------
# Cascade decode over a shared prefix


@dataclass
class SharedPrefix:
    """Python mirror of ``uq_shared_prefix``: pages int32 [num_tokens / 16]
    and lens int32 [batch] on the device."""
    pages: torch.Tensor
    lens: torch.Tensor
    num_tokens: int
    partition_tokens: int = 0

    def c_struct(self):
        return uq_shared_prefix(self.pages.data_ptr(), self.lens.data_ptr(), self.num_tokens, self.partition_tokens)


def cascade_workspace_bytes(num_kv_heads, batch, num_q_heads, max_context, prefix: SharedPrefix, partition_tokens=0):
    sp = prefix.c_struct()
    return int(lib.uq_decode_cascade_workspace_bytes(num_kv_heads, batch, num_q_heads, max_context, partition_tokens,
                                                     ctypes.byref(sp)))


def _prefix(prefix: SharedPrefix, B):
    _need(prefix.pages, "prefix.pages", _I32, (None,), min_numel=max(prefix.num_tokens, 0) // PAGE_SIZE)
    _need(prefix.lens, "prefix.lens", _I32, (B,))


def _cascade_common(q, k_new, v_new, max_context, num_kv_heads, prefix, softmax_scale, partition_tokens, workspace,
                    out, out_dtype):
    B, Hq = _q_out(q, out, HEAD_DIM)
    _prefix(prefix, B)
    if k_new is not None or v_new is not None:
        _new_token(k_new, v_new, B, num_kv_heads)
    if softmax_scale is None:
        softmax_scale = HEAD_DIM ** -0.5
    if workspace is None:
        n = cascade_workspace_bytes(num_kv_heads, B, Hq, max_context, prefix, partition_tokens)
        workspace = torch.empty(n, dtype=torch.uint8, device=q.device)
    _need(workspace, "workspace", _U8)
    if out is None:
        out = torch.empty((B, Hq, HEAD_DIM), dtype=out_dtype, device=q.device)
    ndt = UQ_F32 if k_new is None else _DT[k_new.dtype]
    return B, Hq, softmax_scale, workspace, out, ndt


def decode_cascade(desc: CacheDesc, q, codes, scales, page_table, context_lens, max_context, prefix: SharedPrefix,
                   softmax_scale=None, partition_tokens=0, workspace=None, out=None, out_dtype=torch.float32,
                   k_new=None, v_new=None, stream=None, partials_only=False):
    """Decode attention (or, with k_new/v_new, a decode step) with a shared prefix."""
    B, Hq, scale, workspace, out, ndt = _cascade_common(q, k_new, v_new, max_context, desc.num_kv_heads, prefix,
                                                        softmax_scale, partition_tokens, workspace, out, out_dtype)
    _pools(desc, codes, scales)
    _table(page_table, context_lens, B)
    d = desc.c_struct()
    sp = prefix.c_struct()
    fn = lib.uq_decode_cascade_partials if partials_only else lib.uq_decode_cascade
    st = fn(ctypes.byref(d), _ptr(q), _DT[q.dtype], _ptr(k_new), _ptr(v_new), ndt, B, Hq, _ptr(codes), _ptr(scales),
            _ptr(page_table), page_table.shape[1], _ptr(context_lens), max_context, ctypes.byref(sp), scale,
            partition_tokens, _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_decode_cascade_partials" if partials_only else "uq_decode_cascade")
    return out


def decode_cascade_merge(desc: CacheDesc, batch, num_q_heads, context_lens, max_context, prefix: SharedPrefix,
                         partition_tokens, workspace, out, stream=None):
    _need(context_lens, "context_lens", _I32, (batch,))
    _prefix(prefix, batch)
    _need(workspace, "workspace", _U8)
    _need(out, "out", _OUT, (batch, num_q_heads, HEAD_DIM))
    d = desc.c_struct()
    sp = prefix.c_struct()
    st = lib.uq_decode_cascade_merge(ctypes.byref(d), batch, num_q_heads, _ptr(context_lens), max_context,
                                     ctypes.byref(sp), partition_tokens, _ptr(workspace), workspace.numel(),
                                     _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_decode_cascade_merge")
    return out


def ref_decode_cascade(desc: RefCacheDesc, q, cache, page_table, context_lens, max_context, prefix: SharedPrefix,
                       softmax_scale=None, partition_tokens=0, workspace=None, out=None, out_dtype=torch.float32,
                       k_new=None, v_new=None, stream=None, partials_only=False):
    B, Hq, scale, workspace, out, ndt = _cascade_common(q, k_new, v_new, max_context, desc.num_kv_heads, prefix,
                                                        softmax_scale, partition_tokens, workspace, out, out_dtype)
    _cache(desc, cache)
    _table(page_table, context_lens, B)
    d = desc.c_struct()
    sp = prefix.c_struct()
    fn = lib.uq_ref_decode_cascade_partials if partials_only else lib.uq_ref_decode_cascade
    st = fn(ctypes.byref(d), _ptr(q), _DT[q.dtype], _ptr(k_new), _ptr(v_new), ndt, B, Hq, _ptr(cache),
            _ptr(page_table), page_table.shape[1], _ptr(context_lens), max_context, ctypes.byref(sp), scale,
            partition_tokens, _ptr(workspace), workspace.numel(), _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_ref_decode_cascade_partials" if partials_only else "uq_ref_decode_cascade")
    return out


def ref_decode_cascade_merge(desc: RefCacheDesc, batch, num_q_heads, context_lens, max_context, prefix: SharedPrefix,
                             partition_tokens, workspace, out, stream=None):
    _need(context_lens, "context_lens", _I32, (batch,))
    _prefix(prefix, batch)
    _need(workspace, "workspace", _U8)
    _need(out, "out", _OUT, (batch, num_q_heads, HEAD_DIM))
    d = desc.c_struct()
    sp = prefix.c_struct()
    st = lib.uq_ref_decode_cascade_merge(ctypes.byref(d), batch, num_q_heads, _ptr(context_lens), max_context,
                                         ctypes.byref(sp), partition_tokens, _ptr(workspace), workspace.numel(),
                                         _ptr(out), _DT[out.dtype], _stream(stream))
    _check(st, "uq_ref_decode_cascade_merge")
    return out


# ---------------------------------------------------------------------------
# Measurement probes


def probe_stream_read(buf, sink=None, stream=None):
    """Read every byte of the uint8 tensor ``buf`` once (a plain stream);
    returns the per-block checksum words (int32 [PROBE_STREAM_BLOCKS])."""
    _need(buf, "buf", _U8)
    if sink is None:
        sink = torch.empty(PROBE_STREAM_BLOCKS, dtype=torch.int32, device=buf.device)
    _need(sink, "sink", (torch.int32,), min_numel=PROBE_STREAM_BLOCKS)
    _check(lib.uq_probe_stream_read(_ptr(buf), buf.numel(), _ptr(sink), _stream(stream)), "uq_probe_stream_read")
    return sink


def probe_page_gather(desc: CacheDesc, num_q_heads, codes, scales, page_table, context_lens, max_context,
                      partition_tokens=0, sink=None, stream=None):
    """The FP4 decode kernel's page gather without its arithmetic, for the
    same arguments (head sizes 64, 128, 256); returns the per-wave checksum
    words (4 per block of the launch; an allocated sink holds the bound
    4 x partitions x kv heads x batch)."""
    B = context_lens.shape[0]
    _pools(desc, codes, scales)
    _table(page_table, context_lens, B)
    part = partition_tokens or default_partition(desc, B, num_q_heads, max_context)
    nwords = 4 * max(1, -(-max_context // part)) * desc.num_kv_heads * B
    if sink is None:
        sink = torch.empty(nwords, dtype=torch.int32, device=codes.device)
    _need(sink, "sink", (torch.int32,), min_numel=nwords)
    d = desc.c_struct()
    st = lib.uq_probe_page_gather(ctypes.byref(d), B, num_q_heads, _ptr(codes), _ptr(scales), _ptr(page_table),
                                  page_table.shape[1], _ptr(context_lens), max_context, partition_tokens, _ptr(sink),
                                  sink.numel(), _stream(stream))
    _check(st, "uq_probe_page_gather")
    return sink


def probe_page_gather_cascade(desc: CacheDesc, num_q_heads, codes, scales, page_table, context_lens, max_context,
                              prefix: SharedPrefix, partition_tokens=0, workspace=None, sink=None, stream=None):
    """The cascade decode kernel's page gather without its arithmetic, for
    the same arguments; returns the per-wave checksum words. An allocated
    sink holds an upper bound of the launch's blocks: the context blocks and
    Hkv x ceil(B G / 16) x ceil(prefix tokens / 32) prefix blocks."""
    B = context_lens.shape[0]
    _pools(desc, codes, scales)
    _table(page_table, context_lens, B)
    _prefix(prefix, B)
    if workspace is None:
        n = cascade_workspace_bytes(desc.num_kv_heads, B, num_q_heads, max_context, prefix, partition_tokens)
        workspace = torch.empty(n, dtype=torch.uint8, device=codes.device)
    _need(workspace, "workspace", _U8)
    part = partition_tokens or default_partition(desc, B, num_q_heads, max_context)
    G = num_q_heads // desc.num_kv_heads
    blocks = (max(1, -(-max_context // part)) * desc.num_kv_heads * B
              + desc.num_kv_heads * -(-B * G // 16) * max(1, -(-prefix.num_tokens // 32)))
    if sink is None:
        sink = torch.empty(4 * blocks, dtype=torch.int32, device=codes.device)
    _need(sink, "sink", (torch.int32,), min_numel=1)
    d = desc.c_struct()
    sp = prefix.c_struct()
    st = lib.uq_probe_page_gather_cascade(ctypes.byref(d), B, num_q_heads, _ptr(codes), _ptr(scales),
                                          _ptr(page_table), page_table.shape[1], _ptr(context_lens), max_context,
                                          ctypes.byref(sp), partition_tokens, _ptr(workspace), workspace.numel(),
                                          _ptr(sink), sink.numel(), _stream(stream))
    _check(st, "uq_probe_page_gather_cascade")
    return sink


def probe_mfma(kind, a, b, scale_a=None, scale_b=None, stream=None):
    """n one-wave matrix products: a, b uint8 [n, 64, 32] in the lane layout,
    scale_a, scale_b uint8 [n, 64] (kinds 0, 1, 3) -> float32 [n, 64, 4]."""
    n = a.shape[0]
    _need(a, "a", _U8, (n, 64, 32))
    _need(b, "b", _U8, (n, 64, 32))
    if kind != PROBE_MFMA_BF16:
        _need(scale_a, "scale_a", _U8, (n, 64))
        _need(scale_b, "scale_b", _U8, (n, 64))
    d = torch.empty((n, 64, 4), dtype=torch.float32, device=a.device)
    _check(lib.uq_probe_mfma(kind, _ptr(a), _ptr(b), _ptr(scale_a), _ptr(scale_b), n, _ptr(d), _stream(stream)),
           "uq_probe_mfma")
    return d
