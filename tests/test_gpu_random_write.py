"""Seeded random quantize-on-write cases (uq_quantize_kv) against the
oracle, bit for bit on every pool byte (pools pre-filled with a canary):
head sizes 64/128/256, 1 to 8 KV heads, 0 to 3000 tokens, f32/bf16/f16
rows read as strided K and V views of one fused buffer, physical slots or
logical slots through a page table, padding slots, slots past the pool and
sequences past num_seqs (all skipped), c in {0.1, 0.156, 0.25}, rotate_v,
and rows that are zero or (f32) of magnitude 1e-20 and 1e20.  Each case
prints its parameters first."""
import ctypes

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu

CASES = 32


def params(i):
    rng = np.random.default_rng(7000 + i)
    d = int(rng.choice([64, 128, 256]))
    hkv = int(rng.integers(1, 9))
    T = int(rng.choice([0, 1, 7, int(rng.integers(8, 3001))]))
    dt = [torch.float32, torch.bfloat16, torch.float16][int(rng.integers(0, 3))]
    align = 4 if dt == torch.float32 else 8            # elements per 16 bytes
    pad_mid = align * int(rng.integers(0, 3))
    pad_end = align * int(rng.integers(0, 3))
    paged = bool(rng.random() < 0.5)
    c = float(rng.choice([0.1, 0.156, 0.25]))
    rotate_v = bool(rng.random() < 0.7)
    return dict(d=d, hkv=hkv, T=T, dt=dt, pad_mid=pad_mid, pad_end=pad_end, paged=paged, c=c, rotate_v=rotate_v,
                seed=8000 + i)


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


@pytest.mark.parametrize("i", range(CASES))
def test_random_write(uq, i):
    p = params(i)
    print(f"write case {i}: {p}", flush=True)
    rng = np.random.default_rng(p["seed"])
    d, hkv, T = p["d"], p["hkv"], p["T"]
    row = hkv * d
    num_pages = int(rng.integers(T // 16 + 2, T // 8 + 40))

    # rows: normal, with some tokens zero or of extreme magnitude
    g = torch.Generator().manual_seed(p["seed"])
    buf = torch.randn((T, 2 * row + p["pad_mid"] + p["pad_end"]), generator=g)
    mag = rng.choice([1.0, 0.0, 1e-20, 1e20], size=T, p=[0.85, 0.05, 0.05, 0.05])
    if p["dt"] != torch.float32:
        mag = np.where((mag == 1e-20) | (mag == 1e20), 1.0, mag)
    buf *= torch.as_tensor(mag, dtype=torch.float32)[:, None]
    buf = buf.to(p["dt"])
    k_off, v_off = 0, row + p["pad_mid"]

    # slots: unique physical targets, some padding and some out of range
    if p["paged"]:
        S = min(int(rng.integers(1, 5)), num_pages)
        P = max(1, min(num_pages // 5, num_pages // S))   # S * P <= num_pages
        page_table = rng.permutation(num_pages)[:S * P].reshape(S, P).astype(np.int32)
        logical = rng.permutation(S * P * 16)[:T] if T <= S * P * 16 else None
        if logical is None:
            num_pages = T // 16 + 8
            S, P = 1, num_pages
            page_table = rng.permutation(num_pages).reshape(1, P).astype(np.int32)
            logical = rng.permutation(S * P * 16)[:T]
        slots = logical.astype(np.int64)
        phys = page_table[slots // (P * 16), (slots % (P * 16)) // 16].astype(np.int64) * 16 + slots % 16
        kind = rng.random(T)
        slots = np.where(kind < 0.05, -1 - rng.integers(0, 100, T), slots)                 # padding
        slots = np.where((kind >= 0.05) & (kind < 0.08), S * P * 16 + rng.integers(0, 50, T), slots)  # seq >= S
        phys = np.where(kind < 0.08, -1, phys)
    else:
        page_table = None
        slots = rng.permutation(num_pages * 16)[:T].astype(np.int64)
        kind = rng.random(T)
        slots = np.where(kind < 0.05, -1, slots)
        slots = np.where((kind >= 0.05) & (kind < 0.08), num_pages * 16 + rng.integers(0, 50, T), slots)
        phys = np.where(kind < 0.08, -1, slots)

    dev = torch.device("cuda:0")
    desc = uq.CacheDesc(num_kv_heads=hkv, num_pages=num_pages, c=p["c"], rotate_v=p["rotate_v"], head_dim=d)
    codes, scales = desc.alloc_pools(dev, fill=0xA5)
    if T == 0:
        # zero tokens is a no-op; an empty tensor's pointer is NULL, which the
        # call rejects, so the C ABI gets one-row buffers and num_tokens 0
        one = torch.zeros((1, buf.shape[1]), dtype=p["dt"], device=dev)
        sd = torch.full((1,), 5, dtype=torch.int64, device=dev)
        ptr = lambda t, off=0: ctypes.c_void_p(t.data_ptr() + off)
        st = uq.lib.uq_quantize_kv(ctypes.byref(desc.c_struct()), ptr(one), ptr(one, v_off * one.element_size()),
                                   uq._DT[p["dt"]], 0, buf.shape[1], None, 0, 0, ptr(sd), ptr(codes), ptr(scales),
                                   None)
        assert st == 0
    else:
        bd = buf.to(dev)
        k = bd[:, k_off:k_off + row].unflatten(1, (hkv, d))
        v = bd[:, v_off:v_off + row].unflatten(1, (hkv, d))
        uq.quantize_kv(desc, k, v, torch.as_tensor(slots, device=dev), codes, scales,
                       page_table=None if page_table is None else torch.as_tensor(page_table, device=dev),
                       token_stride=buf.shape[1])
    torch.cuda.synchronize()

    pools = oracle.alloc_pools(num_pages, hkv, fill=0xA5, head_dim=d)
    kf = buf[:, k_off:k_off + row].float().reshape(T, hkv, d).numpy()
    vf = buf[:, v_off:v_off + row].float().reshape(T, hkv, d).numpy()
    oracle.quantize_kv(kf, vf, phys, num_pages, c=p["c"], rotate_v=p["rotate_v"], pools=pools)
    assert np.array_equal(codes.cpu().numpy(), pools[0]), f"case {i}: codes differ"
    assert np.array_equal(scales.cpu().numpy(), pools[1]), f"case {i}: scale bytes differ"
