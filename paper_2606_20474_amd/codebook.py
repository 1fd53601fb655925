"""16-level codebooks for the Ultra-TQ comparison cache (the paper's appendix
"Calibrated LUT int4 KV Encoding (Ultra-TQ)" and section "Calibrated
Centroids").

The keys of that scheme are rotated, divided by their norm and coded to the
nearest of 16 levels.  The paper derives its theoretical levels from the law
of one coordinate of a uniform unit vector in R^d,
(1 + x) / 2 ~ Beta((d-1)/2, (d-1)/2), and prints the largest of them at
d = 64 as 0.342: that is the Lloyd-Max level of N(0, 1) (2.733, Max's table)
scaled by 1/sqrt(d), the Gaussian limit of the law, not the Lloyd-Max level
of the exact law (0.331).  The default codebook follows the printed value.
This module solves both quantizers from closed forms (Lloyd's iteration on
the exact CDF and partial first moment).  A calibrated table (levels refit
on captured keys) is any other ascending list of 16 floats.
"""
from __future__ import annotations

import functools
import math

import numpy as np
from scipy import special, stats


def lloyd_max(cdf, partial_mean, second_moment, levels0, iters=20000):
    """Lloyd's iteration for a density given by closed forms:
    cdf(t) = P(X <= t), partial_mean(t) = E[X; X <= t].  Thresholds are the
    midpoints of the levels, levels the conditional means of their cells.
    Returns (levels, MSE = E[X^2] - sum_k P_k c_k^2)."""
    lv = np.asarray(levels0, np.float64)
    for _ in range(iters):
        t = np.concatenate([[-np.inf], (lv[1:] + lv[:-1]) / 2, [np.inf]])
        lv = np.diff(partial_mean(t)) / np.diff(cdf(t))
    t = np.concatenate([[-np.inf], (lv[1:] + lv[:-1]) / 2, [np.inf]])
    return lv, second_moment - float(np.sum(np.diff(cdf(t)) * lv ** 2))


def gaussian_lloyd_max(n=16):
    """Lloyd-Max quantizer of N(0, 1): (levels, MSE)."""
    return lloyd_max(stats.norm.cdf, lambda t: -stats.norm.pdf(t), 1.0, stats.norm.ppf((np.arange(n) + 0.5) / n))


@functools.lru_cache(maxsize=None)
def _sphere(d: int, n: int):
    a = (d - 1) / 2
    log_z = (2 * a - 1) * math.log(2) + special.betaln(a, a)

    def cdf(t):
        return special.betainc(a, a, np.clip((1 + t) / 2, 0, 1))

    def partial_mean(t):
        # the integral of x (1 - x^2)^(a-1) / Z from -1 to t is -(1 - t^2)^a / (2 a Z)
        u = np.clip(1 - np.square(np.clip(t, -1, 1)), 0, None)
        return -np.exp(a * np.log(np.maximum(u, 1e-300)) - log_z) / (2 * a) * (u > 0)

    lv0 = 2 * special.betaincinv(a, a, (np.arange(n) + 0.5) / n) - 1
    lv, mse = lloyd_max(cdf, partial_mean, 1.0 / d, lv0)
    return tuple(float(x) for x in lv), mse


def sphere_lloyd_max(d: int, n: int = 16):
    """Lloyd-Max quantizer of one coordinate of a uniform unit vector in
    R^d: (levels as float64 array, MSE per coordinate)."""
    lv, mse = _sphere(int(d), int(n))
    return np.array(lv), mse


@functools.lru_cache(maxsize=None)
def _gauss16():
    return tuple(float(x) for x in gaussian_lloyd_max(16)[0])


def default_tq_codebook(d: int = 128) -> np.ndarray:
    """The theoretical (uncalibrated) Ultra-TQ key codebook for head size d:
    the 16 Lloyd-Max levels of N(0, 1) divided by sqrt(d), ascending
    float32."""
    return (np.array(_gauss16()) / math.sqrt(d)).astype(np.float32)
