"""The arithmetic of the matrix instructions the decode kernels are built on,
measured one wave at a time through uq_probe_mfma against exact fp64 sums of
the same decoded operands.

* Operands whose products and sums are exact in fp32 must come back exact:
  this pins the lane layouts, nibble order and scale placement the kernels
  assume (a transposed operand or a scale on the wrong k-block fails it).
* Random operands bound each instruction's error relative to the largest
  product of the dot product, for operands like the kernel's and for
  arbitrary ones.  These bounds are what the tolerances of the other tests
  rest on: the FP4 x FP8 form (the QK^T of the FP4 cache), whose
  error enters the bound derived in test_gpu_qk_precision_bound.py; the FP8 x FP8 form (the FP8-KV comparator's
  QK^T), which sets that comparator's tolerance in test_gpu_ref_caches.py;
  and the BF16 form of PV.
"""
import numpy as np
import pytest
import torch

pytestmark = pytest.mark.gpu

E2M1 = np.array([0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0])   # the FP4 grid F (section "Dequantization")

# Largest error / largest |product| of the dot product, per instruction and
# operand class (measured maxima over such draws in the comments):
#   "kernel": FP8 operands rounded from N(0, 1) values (the decode kernel's
#             rotated query), random E2M1 codes, block scales 2^-7 .. 2^7
#             (the per-group scales of one cache row stay in a narrow band);
#   "any":    random FP8 bytes over the whole E4M3 range, block scales
#             2^-17 .. 2^18.
# FP4 x FP8 returns the exactly rounded sum on most kernel-like dot products
# (85-100 %), but not on all.
BOUND = {(0, "kernel"): 2.0 ** -12.5,   # 2^-14.0
         (0, "any"): 2.0 ** -10.5,      # 2^-10.9
         (1, "kernel"): 2.0 ** -11.5,   # 2^-11.8
         (1, "any"): 2.0 ** -10.5,      # 2^-11.1
         (2, "kernel"): 2.0 ** -19,     # 2^-21
         (2, "any"): 2.0 ** -19,
         (3, "kernel"): 2.0 ** -12.5,   # 2^-13.0
         (3, "any"): 2.0 ** -10.5}      # 2^-11.0


@pytest.fixture(scope="module")
def uq():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import uq as mod
    return mod


def log(msg):
    print(msg, flush=True)


def e2m1_decode(codes):
    v = E2M1[codes & 7]
    return np.where(codes & 8, -v, v)


def e4m3_decode(b):
    return torch.from_numpy(np.ascontiguousarray(b, dtype=np.uint8)).view(torch.float8_e4m3fn).double().numpy()


def fp4_operand(codes):
    """codes [n, 16 rows, 128 k] (4-bit) -> lane bytes [n, 64, 32]: lane 16 j + i
    holds row i, k 32 j .. 32 j + 31, two codes per byte, low nibble first."""
    n = codes.shape[0]
    out = np.zeros((n, 64, 32), np.uint8)
    for j in range(4):
        blk = codes[:, :, 32 * j:32 * j + 32]
        out[:, 16 * j:16 * j + 16, :16] = (blk[:, :, 0::2] | (blk[:, :, 1::2] << 4)).astype(np.uint8)
    return out


def fp8_operand(bytes_):
    """bytes [n, 16, 128] -> lane bytes: lane 16 g + i holds row i, k 16 g ..
    16 g + 15 in bytes 0..15 and k 64 + 16 g .. in bytes 16..31."""
    n = bytes_.shape[0]
    out = np.zeros((n, 64, 32), np.uint8)
    for g in range(4):
        out[:, 16 * g:16 * g + 16, :16] = bytes_[:, :, 16 * g:16 * g + 16]
        out[:, 16 * g:16 * g + 16, 16:] = bytes_[:, :, 64 + 16 * g:64 + 16 * g + 16]
    return out


def bf16_operand(vals):
    """values [n, 16, 32] (exact BF16) -> lane bytes: lane 16 g + i holds row i,
    k 8 g .. 8 g + 7."""
    n = vals.shape[0]
    bits = torch.from_numpy(vals.astype(np.float32)).bfloat16().view(torch.int16).numpy().view(np.uint16)
    out = np.zeros((n, 64, 32), np.uint8)
    for g in range(4):
        out[:, 16 * g:16 * g + 16, :16] = np.ascontiguousarray(bits[:, :, 8 * g:8 * g + 8]).view(np.uint8)
    return out


def scale_lanes(s):
    """scale bytes [n, 16 rows, 4 k-blocks] -> [n, 64]: lane 16 j + i."""
    return np.ascontiguousarray(s.transpose(0, 2, 1).reshape(s.shape[0], 64)).astype(np.uint8)


def unlane(d):
    """[n, 64, 4] -> D [n, 16, 16]: lane l element r is D[4 (l / 16) + r][l % 16]."""
    n = d.shape[0]
    out = np.zeros((n, 16, 16))
    for l in range(64):
        for r in range(4):
            out[:, 4 * (l // 16) + r, l % 16] = d[:, l, r]
    return out


def run(uq, kind, a, b, sa=None, sb=None):
    dev = torch.device("cuda:0")
    t = lambda x: None if x is None else torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    d = uq.probe_mfma(kind, t(a), t(b), t(sa), t(sb))
    torch.cuda.synchronize()
    return unlane(d.cpu().numpy().astype(np.float64))


def case(rng, kind, n, exact, cls="any"):
    """Operands of `kind`: returns (lane a, lane b, lane scales a, b, exact D,
    largest |product| per output)."""
    if kind == 2:
        if exact:   # small integers: every product and sum exact in fp32
            A = rng.integers(-8, 9, (n, 16, 32)).astype(np.float64)
            B = rng.integers(-8, 9, (n, 32, 16)).astype(np.float64)
        else:
            A = torch.from_numpy(rng.standard_normal((n, 16, 32))).bfloat16().double().numpy()
            B = torch.from_numpy(rng.standard_normal((n, 32, 16)) * np.exp(rng.standard_normal((n, 32, 16)))
                                 ).bfloat16().double().numpy()
        a = bf16_operand(A)
        b = bf16_operand(B.transpose(0, 2, 1))
        prod = A[:, :, :, None] * B[:, None, :, :]
        return a, b, None, None, prod.sum(axis=2), np.abs(prod).max(axis=2)
    # k = 128, scaled: A rows x k, B k x columns
    fp4_a, fp4_b = kind == 0, kind == 3
    if exact:
        # scales 2^-1 .. 2^1: products are multiples of 2^-3 below 2^8, so the
        # sums are exact even for an accumulator that keeps only the top ~14
        # bits of the largest product
        lo, hi = 126, 128
    elif cls == "kernel":
        lo, hi = 120, 134
    else:
        lo, hi = 110, 145
    sa = rng.integers(lo, hi + 1, (n, 16, 4))
    sb = rng.integers(lo, hi + 1, (n, 16, 4))

    def draw(fp4):
        if fp4:
            codes = rng.integers(0, 16, (n, 16, 128))
            return codes, e2m1_decode(codes)
        if exact:   # E4M3 bytes of small integers 0..8 with a sign: exact products
            x = rng.integers(-8, 9, (n, 16, 128)).astype(np.float32)
            byts = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        elif cls == "kernel":
            x = rng.standard_normal((n, 16, 128)).astype(np.float32)
            byts = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        else:
            byts = rng.integers(0, 256, (n, 16, 128)).astype(np.uint8)
            byts[(byts & 0x7F) == 0x7F] = 0     # no NaN
        return byts, e4m3_decode(byts)
    ra, va = draw(fp4_a)
    rb, vb = draw(fp4_b)
    a = fp4_operand(ra) if fp4_a else fp8_operand(ra)
    b = fp4_operand(rb) if fp4_b else fp8_operand(rb)
    ka = np.repeat(2.0 ** (sa.astype(np.float64) - 127), 32, axis=2)   # [n, 16, 128]
    kb = np.repeat(2.0 ** (sb.astype(np.float64) - 127), 32, axis=2)
    A = va * ka                       # [n, rows, k]
    B = (vb * kb).transpose(0, 2, 1)  # [n, k, columns]
    prod = A[:, :, :, None] * B[:, None, :, :]
    return a, b, scale_lanes(sa), scale_lanes(sb), prod.sum(axis=2), np.abs(prod).max(axis=2)


NAMES = {0: "scaled 16x16x128 FP4 x FP8", 1: "scaled 16x16x128 FP8 x FP8", 2: "16x16x32 BF16",
         3: "scaled 16x16x128 FP8 x FP4"}


@pytest.mark.parametrize("kind", [0, 1, 2, 3])
def test_exact_sums_come_back_exact(uq, kind):
    """Sums exact in fp32 return exactly: the lane layouts, nibble order and
    the scale byte of (row or column i, k-block j) at lane 16 j + i are the
    ones the kernels use."""
    rng = np.random.default_rng(100 + kind)
    a, b, sa, sb, ref, _ = case(rng, kind, 256, exact=True)
    got = run(uq, kind, a, b, sa, sb)
    log(f"{NAMES[kind]}: exact-sum cases, max |error| {np.abs(got - ref).max():.3e}")
    assert np.array_equal(got, ref)


@pytest.mark.parametrize("cls", ["kernel", "any"])
@pytest.mark.parametrize("kind", [0, 1, 2, 3])
def test_error_relative_to_largest_product(uq, kind, cls):
    """Random operands of a class: |D - exact| <= bound x max |product| of
    that dot product (and the result is finite)."""
    rng = np.random.default_rng(200 + 10 * kind + (cls == "any"))
    a, b, sa, sb, ref, pmax = case(rng, kind, 1024, exact=False, cls=cls)
    got = run(uq, kind, a, b, sa, sb)
    assert np.all(np.isfinite(got))
    err = np.abs(got - ref)
    rel = err / np.maximum(pmax, 1e-300)
    rounded = ref.astype(np.float32).astype(np.float64)
    bound = BOUND[(kind, cls)]
    log(f"{NAMES[kind]}, {cls} operands: exactly rounded {np.mean(got == rounded) * 100:.1f} %, max error / "
        f"max |product| 2^{np.log2(max(rel.max(), 2.0 ** -60)):.1f} (bound 2^{np.log2(bound):.1f})")
    assert rel.max() <= bound
