"""Offline fit of the scale constant c (section "Constant-Optimized Scaling").

The encoder maps each group of 32 rotated channels with absmax m onto the
E2M1 grid with the scale s = c m, rounded in the cache to the power of two
2^round(log2(c m)).  c is one global constant, chosen once to minimise the
round-trip error E[(z - s q(z / s))^2] on rotated key rows.  This module
sweeps and fits c with the GPU encoder (``uq_quantize_error``: the same
rotation, exponent rule and hardware E2M1 conversion as the cache writer),
under either scale rule:

  * ``pow2=False``: the continuous s = c m of the paper's objective;
  * ``pow2=True``: the cache's own 2^round(log2(c m)).

Command line (synthetic rows; pass real keys through :func:`fit_c`)::

    python -m paper_2606_20474_amd.calibrate --source unit --dim 128 --rows 262144
"""
from __future__ import annotations

import argparse
import json

import numpy as np
import torch

from . import uq
from . import workloads


def round_trip_error(x, c_values, rotate=True, pow2=True, chunk_rows=1 << 22, stream=None) -> np.ndarray:
    """Sums (squared error, energy) per c over all rows of x [N, 128] on the
    device, in row chunks of ``chunk_rows``; float64 [len(c), 2]."""
    c = torch.as_tensor(np.asarray(c_values, np.float32), device=x.device)
    rows = x.reshape(-1, uq.HEAD_DIM)
    sums = torch.zeros((c.numel(), 2), dtype=torch.float64, device=x.device)
    for lo in range(0, rows.shape[0], chunk_rows):
        uq.quantize_error(rows[lo:lo + chunk_rows], c, rotate, pow2, sums, stream)
    return sums.cpu().numpy()


def relative_mse(x, c_values, rotate=True, pow2=True) -> np.ndarray:
    """E|z - s q(z/s)|^2 / E|z|^2 per c."""
    s = round_trip_error(x, c_values, rotate, pow2)
    return s[:, 0] / s[:, 1]


def fit_c(x, lo=0.05, hi=0.5, points=46, rounds=3, rotate=True, pow2=False):
    """Grid search for the minimiser over [lo, hi], refined ``rounds`` times
    around the best point (one launch per round).  Returns (c, relative MSE,
    the last grid, its MSE curve)."""
    for _ in range(rounds):
        grid = np.linspace(lo, hi, points, dtype=np.float32)
        r = relative_mse(x, grid, rotate, pow2)
        i = int(np.argmin(r))
        lo, hi = float(grid[max(i - 1, 0)]), float(grid[min(i + 1, points - 1)])
    return float(grid[i]), float(r[i]), grid, r


def synthetic_rows(source: str, rows: int, dim: int, seed: int, device) -> tuple[torch.Tensor, bool]:
    """(rows [N, 128] on the device, rotate): uniform unit vectors of R^dim
    packed 128 channels a row (already rotated: a uniform vector stays
    uniform under any rotation), or key rows of the cache recipe (rotated by
    the encoder)."""
    if source == "unit":
        if dim % 32 or (dim > 128 and dim % 128) or (dim < 128 and 128 % dim):
            raise ValueError("dim must be 32, 64, 128 or a multiple of 128")
        n = max(rows * 128 // dim, 1)
        return torch.as_tensor(workloads.unit_vectors(n, dim, seed).reshape(-1, 128), device=device), False
    if source == "keys":
        return torch.as_tensor(workloads.key_rows(rows, seed), device=device), True
    raise ValueError(source)


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--source", choices=["unit", "keys"], default="unit")
    ap.add_argument("--dim", type=int, default=128, help="vector length of the unit vectors")
    ap.add_argument("--rows", type=int, default=1 << 18)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--constants", default="0.156,0.195,1.0")
    args = ap.parse_args(argv)
    if not torch.cuda.is_available():
        raise SystemExit("the calibration runs the GPU encoder; no GPU is visible")
    x, rotate = synthetic_rows(args.source, args.rows, args.dim, args.seed, torch.device("cuda:0"))
    consts = [float(c) for c in args.constants.split(",")]
    report = {"source": args.source, "dim": args.dim, "rows": int(x.shape[0]), "rotate": rotate}
    # time one sweep of 46 constants per scale rule (after one untimed call)
    grid = np.linspace(0.05, 0.5, 46, dtype=np.float32)
    for pow2 in (False, True):
        round_trip_error(x, grid, rotate, pow2)
        t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        t0.record()
        round_trip_error(x, grid, rotate, pow2)
        t1.record()
        t1.synchronize()
        ms = t0.elapsed_time(t1)
        report["sweep46_ms_pow2" if pow2 else "sweep46_ms_continuous"] = round(ms, 3)
    for pow2 in (False, True):
        key = "pow2" if pow2 else "continuous"
        c, r, _, _ = fit_c(x, rotate=rotate, pow2=pow2)
        report[key] = {"argmin_c": round(c, 4), "rel_mse": r,
                       "at": dict(zip(map(str, consts), map(float, relative_mse(x, consts, rotate, pow2))))}
    print(json.dumps(report))


if __name__ == "__main__":
    main()
