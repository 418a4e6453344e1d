"""Offline cost calibration (fp64 CAEE oracle) -- TEST INFRASTRUCTURE ONLY.

Sec. IV-A calibrates the per-expert cost of moving S_e bytes over the data
path of device d as

    C~(e, d) = alpha_d * S_e / B_d + beta_d,

with B_d the nominal bandwidth, alpha_d the measured degradation factor and
beta_d a fixed per-transfer overhead.  Given measured times t_i of moving
S_i bytes, the calibration is the ordinary least-squares line of t on
x = S / B, written here in its closed form:

    alpha = sum (x_i - mean x)(t_i - mean t) / sum (x_i - mean x)^2,
    beta  = mean t - alpha * mean x.

When the transfers are timed in groups (m experts per kernel call, plus one
fixed launch cost c0 per call), the model of a call is
    t = c0 + m * (alpha * S / B + beta),
a linear least-squares problem in (alpha, beta, c0) solved here from its
normal equations.
"""
from __future__ import annotations

import numpy as np


def fit_alpha_beta(sizes_bytes, times, bandwidth):
    """Closed-form least-squares (alpha, beta) of t = alpha * S / B + beta."""
    x = np.asarray(sizes_bytes, dtype=np.float64) / float(bandwidth)
    t = np.asarray(times, dtype=np.float64)
    if x.size < 2 or np.all(x == x[0]):
        raise ValueError("at least two distinct sizes are needed")
    xm, tm = x.mean(), t.mean()
    alpha = float(np.sum((x - xm) * (t - tm)) / np.sum((x - xm) ** 2))
    beta = float(tm - alpha * xm)
    return alpha, beta


def fit_grouped(counts, sizes_bytes, times, bandwidth):
    """(alpha, beta, c0) of t = c0 + m * (alpha * S / B + beta) by the normal
    equations of the least-squares problem."""
    m = np.asarray(counts, dtype=np.float64)
    x = np.asarray(sizes_bytes, dtype=np.float64) / float(bandwidth)
    t = np.asarray(times, dtype=np.float64)
    A = np.stack([m * x, m, np.ones_like(m)], axis=1)
    theta = np.linalg.solve(A.T @ A, A.T @ t)
    return float(theta[0]), float(theta[1]), float(theta[2])


def cost_of(sizes_bytes, alpha, beta, bandwidth):
    """C~ for each size (same unit as the times the fit was made from)."""
    return alpha * np.asarray(sizes_bytes, dtype=np.float64) / float(bandwidth) + beta
