"""Pins of the oracle at head sizes 64 and 256 (the FP4 format of Algorithm 1
with d/32 groups per vector and an d-point rotation; the paper's head size
is 128, and its codebook analysis also covers 64 and 256).

Against routes other than the oracle's own formulas: scipy's Sylvester
Hadamard matrix, numpy's log2 for the exponent window, brute-force nearest
levels, hand-derived layout offsets (tests/golden/page_layout_hd.txt),
scipy's softmax and invariants; and the 128 entry points equal the
head-size ones at d = 128.
"""
import math
import os

import numpy as np
import pytest
import scipy.linalg
import scipy.special

import oracle

RNG = np.random.default_rng(64256)
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])


@pytest.mark.parametrize("d", [64, 256])
def test_rotation_is_the_scaled_sylvester_matrix(d):
    H = scipy.linalg.hadamard(d).astype(np.float64) / math.sqrt(d)
    for _ in range(4):
        x = RNG.standard_normal(d)
        np.testing.assert_allclose(oracle.wht_f64(x), H @ x, rtol=0, atol=1e-12)
        xf = x.astype(np.float32)
        np.testing.assert_allclose(oracle.wht_f32(xf).astype(np.float64), H @ xf.astype(np.float64), rtol=0,
                                   atol=1e-5 * np.abs(xf).sum() / math.sqrt(d))
    y = oracle.wht_f64(oracle.wht_f64(x))
    np.testing.assert_allclose(y, x, atol=1e-12)


def test_128_entry_points_equal_the_head_size_ones():
    x = RNG.standard_normal((5, 128)).astype(np.float32)
    assert np.array_equal(oracle.wht128_f32(x), oracle.wht_f32(x))
    lib = oracle.lib()
    c1 = np.empty(128, np.uint8)
    s1 = np.empty(4, np.uint8)
    lib.uqo_quantize_vector(oracle._ptr(x[0]), np.float32(0.156), 1, oracle._ptr(c1), oracle._ptr(s1))
    c2, s2 = oracle.quantize_vector(x[0])
    assert np.array_equal(c1, c2) and np.array_equal(s1, s2)


@pytest.mark.parametrize("d", [64, 256])
def test_quantize_vector_groups_and_codes(d):
    for _ in range(50):
        x = (RNG.standard_normal(d) * 10 ** RNG.uniform(-3, 3)).astype(np.float32)
        codes, sb = oracle.quantize_vector(x, rotate=True)
        assert codes.shape == (d,) and sb.shape == (d // 32,)
        z = oracle.wht_f32(x).astype(np.float64)
        for g in range(d // 32):
            m = np.abs(z[32 * g:32 * g + 32]).max()
            E = int(sb[g]) - 127
            r = float(np.float32(np.float32(0.156) * np.float32(m))) / 2.0 ** E
            assert 2 ** -0.5 <= r < 2 ** 0.5
            t = z[32 * g:32 * g + 32] / 2.0 ** E
            near = np.argmin(np.abs(np.abs(t)[:, None] - E2M1[None, :]), axis=1)
            got = codes[32 * g:32 * g + 32] & 7
            ties = np.min(np.abs(np.abs(t)[:, None] - (E2M1[1:] + E2M1[:-1])[None, :] / 2), axis=1) < 1e-12
            assert np.all((got == near) | ties | (np.abs(t) > 5))
            assert np.all(got[np.abs(t) > 5] == 7)


def test_layout_spot_values():
    rows = [r.split("#")[0].split() for r in open(os.path.join(GOLDEN, "page_layout_hd.txt"))]
    for d, kind, t, c, byte, nib in [(int(r[0]), r[1], int(r[2]), int(r[3]), int(r[4]), r[5]) for r in rows if r]:
        pools = oracle.alloc_pools(1, 1, head_dim=d)
        k = np.zeros(d, np.float32)
        v = np.zeros(d, np.float32)
        e = np.zeros(d)
        e[c] = 1.0
        if kind == "K":
            k = oracle.wht_f64(e).astype(np.float32)      # rotates back to e_c
        else:
            v = e.astype(np.float32)
        oracle.quantize_kv(k[None, None], v[None, None], [t], 1, rotate_v=False, pools=pools)
        codes, scales = pools
        if kind == "S":
            # V scale byte of group c // 32 for token t: the V tile's scales follow the K tile's
            assert scales[d // 2 + byte] == 127 - 3, (d, t, c, scales[d // 2 + byte])
            continue
        base = 0 if kind == "K" else 8 * d
        b = codes[base + byte]
        code = (b >> 4) if nib == "hi" else (b & 15)
        assert code == 7, (d, kind, t, c, byte, code)


@pytest.mark.parametrize("d", [64, 256])
def test_layout_is_a_bijection(d):
    seen = set()
    for t in range(16):
        for c in range(d):
            pools = oracle.alloc_pools(1, 1, head_dim=d)
            v = np.zeros((1, 1, d), np.float32)
            v[0, 0, c] = 1.0
            oracle.quantize_kv(np.zeros_like(v), v, [t], 1, rotate_v=False, pools=pools)
            nz = np.nonzero(pools[0][8 * d:])[0]
            assert nz.size == 1
            seen.add((int(nz[0]), "hi" if pools[0][8 * d + nz[0]] >> 4 else "lo"))
    assert len(seen) == 16 * d


def naive_attention(q, pools, pt, ctx, hkv, scale, rotate_v, d):
    B, Hq, _ = q.shape
    G = Hq // hkv
    out = np.zeros((B, Hq, d))
    for b in range(B):
        for h in range(Hq):
            if ctx[b] == 0:
                continue
            q8 = np.array([oracle.e4m3_value(x) for x in oracle.prepare_query(q[b, h])])
            K = np.array([oracle.dequant_vector(pools, hkv, pt[b, j // 16], h // G, 0, j % 16, d) for j in range(ctx[b])])
            V = np.array([oracle.dequant_vector(pools, hkv, pt[b, j // 16], h // G, 1, j % 16, d) for j in range(ctx[b])])
            o = scipy.special.softmax(scale * K @ q8) @ V
            if rotate_v:
                o = scipy.linalg.hadamard(d) @ o / math.sqrt(d)
            out[b, h] = o
    return out


@pytest.mark.parametrize("d", [64, 256])
@pytest.mark.parametrize("rotate_v", [True, False])
def test_attention_brute_force(d, rotate_v):
    B, Hq, Hkv, P = 2, 4, 2, 5
    ctx = np.array([29, 0], np.int32)
    pt = np.array([[3, 0], [1, 2]], np.int32)
    T = 32
    k = RNG.standard_normal((T, Hkv, d)).astype(np.float32)
    v = RNG.standard_normal((T, Hkv, d)).astype(np.float32)
    slots = np.array([pt[0, j // 16] * 16 + j % 16 for j in range(T)])
    pools = oracle.quantize_kv(k, v, slots, P, rotate_v=rotate_v, pools=oracle.alloc_pools(P, Hkv, head_dim=d))
    q = RNG.standard_normal((B, Hq, d)).astype(np.float32)
    scale = 1 / math.sqrt(d)
    got = oracle.decode_attention(q, pools, pt, ctx, Hkv, scale, rotate_v)
    ref = naive_attention(q, pools, pt, ctx, Hkv, scale, rotate_v, d)
    np.testing.assert_allclose(got, ref, rtol=0, atol=1e-10)
    assert np.all(got[1] == 0)


@pytest.mark.parametrize("d", [64, 256])
def test_attention_identical_keys_average_the_values(d):
    T = 20
    k = np.tile(RNG.standard_normal(d).astype(np.float32), (T, 1, 1))
    v = RNG.standard_normal((T, 1, d)).astype(np.float32)
    pools = oracle.quantize_kv(k, v, np.arange(T), 2, rotate_v=False, pools=oracle.alloc_pools(2, 1, head_dim=d))
    q = RNG.standard_normal((1, 2, d)).astype(np.float32)
    out = oracle.decode_attention(q, pools, np.array([[0, 1]], np.int32), np.array([T], np.int32), 1, None, False)
    vmean = np.mean([oracle.dequant_vector(pools, 1, t // 16, 0, 1, t % 16, d) for t in range(T)], axis=0)
    np.testing.assert_allclose(out[0, 0], vmean, atol=1e-12)
    np.testing.assert_allclose(out[0, 1], vmean, atol=1e-12)
