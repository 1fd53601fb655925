"""The GPU round-trip error (uq_quantize_error) and the c fit built on it
(paper_2606_20474_amd.calibrate), against the oracle.

The sums compare with oracle.quantize_error on the same rows: the codes are
decided in fp32 on both sides (the oracle's nearest-level search and the
hardware E2M1 conversion agree on every probe case), the sums differ only by
fp32 versus fp64 accumulation, so the relative difference bound is 1e-5 for
the error and 1e-6 for the energy.  Cases: f32 and bf16 rows, strided rows,
both scale rules, with and without the rotation, a ragged row count, two
calls accumulating, an empty call; the fit on unit vectors and on key rows;
and a 4M-row call (the energy equals the inputs' sum of squares, the
rotation being orthonormal; the relative MSE matches the oracle's on a
sample).
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2606_20474_amd import workloads

pytestmark = pytest.mark.gpu

C_LIST = [0.1, 0.156, 0.195, 0.25, 1.0]


@pytest.fixture(scope="module")
def mods():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2606_20474_amd import calibrate, uq
    return uq, calibrate


def log(msg):
    print(msg, flush=True)


def close(got, ref, what):
    got, ref = np.asarray(got), np.asarray(ref)
    e = np.abs(got[:, 0] - ref[:, 0]) / ref[:, 0]
    t = np.abs(got[:, 1] - ref[:, 1]) / ref[:, 1]
    log(f"{what}: error rel-diff {e.max():.2e}, energy rel-diff {t.max():.2e}")
    assert e.max() <= 1e-5, (what, e)
    assert t.max() <= 1e-6, (what, t)


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("rotate", [True, False])
@pytest.mark.parametrize("pow2", [True, False])
def test_error_against_oracle(mods, dtype, rotate, pow2):
    uq, _ = mods
    dev = torch.device("cuda:0")
    log(f"quantize_error {dtype} rotate={rotate} pow2={pow2}")
    x = torch.as_tensor(workloads.key_rows(1000, seed=41)).to(dtype)
    got = uq.quantize_error(x.to(dev), torch.tensor(C_LIST), rotate, pow2)
    ref = oracle.quantize_error(x.float().numpy(), C_LIST, rotate, pow2)
    close(got.cpu().numpy(), ref, f"{dtype} rotate={rotate} pow2={pow2}")


def test_strided_rows_and_accumulation(mods):
    """K rows of a [T, 2, 128] tensor (row stride 256), in two calls into
    the same sums, and an empty call that leaves them alone."""
    uq, _ = mods
    dev = torch.device("cuda:0")
    kv = torch.as_tensor(workloads.key_rows(2 * 777, seed=42)).reshape(777, 2, 128).to(torch.bfloat16)
    k = kv.to(dev)[:, 0, :]
    assert k.stride(0) == 256
    c = torch.tensor(C_LIST)
    sums = uq.quantize_error(k[:300], c)
    uq.quantize_error(k[300:], c, sums=sums)
    uq.quantize_error(k[:0], c, sums=sums)
    ref = oracle.quantize_error(kv[:, 0, :].float().numpy(), C_LIST)
    close(sums.cpu().numpy(), ref, "strided, two calls")


def test_fit_on_unit_vectors(mods):
    """The minimiser on uniform unit vectors of R^128: near 0.16 for the
    continuous scale, near 0.195 for the power-of-two scale; the GPU curve
    and the oracle's pick the same grid point or a neighbour."""
    uq, calibrate = mods
    dev = torch.device("cuda:0")
    u = workloads.unit_vectors(65536, 128, seed=43)
    x = torch.as_tensor(u, device=dev)
    grid = np.round(np.arange(0.140, 0.2205, 0.004), 3).astype(np.float32)
    for pow2, lo, hi in ((False, 0.150, 0.170), (True, 0.186, 0.204)):
        c, r, _, _ = calibrate.fit_c(x, rotate=False, pow2=pow2)
        log(f"fit pow2={pow2}: c={c:.4f} rel-MSE {r:.5f}")
        assert lo <= c <= hi
        g = calibrate.relative_mse(x, grid, rotate=False, pow2=pow2)
        o = oracle.quantize_error(u[:16384], grid, rotate=False, pow2=pow2)
        o = o[:, 0] / o[:, 1]
        assert abs(int(np.argmin(g)) - int(np.argmin(o))) <= 1
        assert g[np.argmin(np.abs(grid - 0.156))] == pytest.approx(o[np.argmin(np.abs(grid - 0.156))], rel=0.02)


def test_fit_on_key_rows(mods):
    """Key rows of the cache recipe, rotated by the encoder: the fit and the
    oracle agree on the minimiser's grid neighbourhood."""
    uq, calibrate = mods
    dev = torch.device("cuda:0")
    k = workloads.key_rows(32768, seed=44)
    x = torch.as_tensor(k, device=dev)
    grid = np.round(np.arange(0.10, 0.30, 0.005), 3).astype(np.float32)
    for pow2 in (False, True):
        g = calibrate.relative_mse(x, grid, rotate=True, pow2=pow2)
        o = oracle.quantize_error(k, grid, rotate=True, pow2=pow2)
        o = o[:, 0] / o[:, 1]
        log(f"keys pow2={pow2}: GPU argmin {grid[np.argmin(g)]}, oracle argmin {grid[np.argmin(o)]}")
        assert abs(int(np.argmin(g)) - int(np.argmin(o))) <= 1
        assert np.allclose(g, o, rtol=1e-5)


def test_large_call(mods):
    """4M bf16 key rows (1 GiB) in one call."""
    uq, _ = mods
    dev = torch.device("cuda:0")
    n = 1 << 22
    g = torch.Generator(device=dev).manual_seed(45)
    x = torch.randn((n, 128), generator=g, device=dev).to(torch.bfloat16)
    log("quantize_error 4M rows")
    sums = uq.quantize_error(x, torch.tensor(C_LIST), rotate=True, pow2=True).cpu().numpy()
    energy = float(x.double().square().sum())
    assert sums[:, 1] == pytest.approx(energy, rel=1e-5)
    sample = x[:: 256].float().cpu().numpy()
    ref = oracle.quantize_error(sample, C_LIST, rotate=True, pow2=True)
    assert np.allclose(sums[:, 0] / sums[:, 1], ref[:, 0] / ref[:, 1], rtol=0.02)
