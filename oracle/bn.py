"""Batch normalisation in training mode (batch statistics), per channel of an
NHWC tensor, and its vector-Jacobian product.

The paper's residual functions are conv-BN-ReLU stacks (ResNet/RevNet blocks,
Sec. 4.1 "Model adaptations").  Readings where the paper is silent:
  * epsilon = 1e-5 and running-statistics momentum 0.1;
  * the normalisation uses the biased batch variance, the running variance
    is fed the unbiased one (m / (m - 1));
  * running statistics are updated only while the activations are recomputed
    during the backward pass, never in the forward (Sec. 4.1).
"""
from __future__ import annotations

import numpy as np

AXES = (0, 1, 2)


def forward(h: np.ndarray, gamma: np.ndarray, beta: np.ndarray, eps: float):
    """Returns (out, cache) with cache = (xhat, rstd, mean, var)."""
    mean = h.mean(axis=AXES)
    var = ((h - mean) ** 2).mean(axis=AXES)
    rstd = 1.0 / np.sqrt(var + eps)
    xhat = (h - mean) * rstd
    return gamma * xhat + beta, (xhat, rstd, mean, var)


def backward(d: np.ndarray, cache, gamma: np.ndarray):
    """VJP of forward(): returns (dh, dgamma, dbeta)."""
    xhat, rstd, _, _ = cache
    m = d.shape[0] * d.shape[1] * d.shape[2]
    dbeta = d.sum(axis=AXES)
    dgamma = (d * xhat).sum(axis=AXES)
    dh = (gamma * rstd) * (d - dbeta / m - xhat * (dgamma / m))
    return dh, dgamma, dbeta


def running_update(run_mean: np.ndarray, run_var: np.ndarray, cache, m: int, momentum: float):
    """Exponential running statistics (unbiased variance), returned as new arrays."""
    _, _, mean, var = cache
    new_mean = (1.0 - momentum) * run_mean + momentum * mean
    new_var = (1.0 - momentum) * run_var + momentum * var * (m / (m - 1.0))
    return new_mean, new_var
