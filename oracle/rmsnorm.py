"""Float64 RMSNorm, the final normalisation of the mask predictor's hidden
states before the LM head (the h of log p_theta(y | y_t, x) in Eq.
per_step_loss is the norm's output).

TEST INFRASTRUCTURE: part of the oracle; see ``oracle/__init__.py``.

  r      = (mean_i x_i^2 + eps)^(-1/2)          per row
  h_i    = gamma_i x_i r

The LM head is a bf16 product, so its input is the norm's output rounded to
bfloat16 (``round_to_bf16``: 8 significant bits, round to nearest, ties to
even); the rounding is passed through unchanged in the backward.

Backward, from the definition (dr/dx_k = -r^3 x_k / d):

  dx_k     = r gamma_k dh_k - (r^3 / d) x_k sum_i gamma_i dh_i x_i
  dgamma_i = sum over rows of dh_i x_i r
"""
from __future__ import annotations

import numpy as np


def rmsnorm(x: np.ndarray, gamma: np.ndarray, eps: float):
    """h = gamma * x / sqrt(mean(x^2) + eps) over the last axis; returns (h, r)."""
    x = np.asarray(x, dtype=np.float64)
    r = 1.0 / np.sqrt(np.mean(x * x, axis=-1, keepdims=True) + eps)
    return x * r * np.asarray(gamma, dtype=np.float64), r


def rmsnorm_backward(x: np.ndarray, gamma: np.ndarray, eps: float, dh: np.ndarray):
    """(dx, dgamma) for upstream gradient dh of the same shape as x (rows on
    all leading axes); dgamma is summed over every row."""
    x = np.asarray(x, dtype=np.float64)
    gamma = np.asarray(gamma, dtype=np.float64)
    d = x.shape[-1]
    _, r = rmsnorm(x, gamma, eps)
    proj = np.sum(gamma * dh * x, axis=-1, keepdims=True)
    dx = r * gamma * dh - (r ** 3 / d) * x * proj
    dgamma = np.sum((dh * x * r).reshape(-1, d), axis=0)
    return dx, dgamma


def round_to_bf16(v: np.ndarray) -> np.ndarray:
    """Nearest bfloat16 value (8 significant bits, ties to even) of float64 v,
    returned as float64 (normal range; the values here never leave it)."""
    v = np.asarray(v, dtype=np.float64)
    m, e = np.frexp(v)                       # v = m 2^e, |m| in [0.5, 1)
    return np.ldexp(np.rint(m * 256.0) / 256.0, e)
