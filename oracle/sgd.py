"""SGD with momentum (Nesterov by default) and gradient accumulation.

Sec. 4.1 (experimental setup): SGD with Nesterov momentum 0.9; no weight
decay on BN parameters or biases; accumulated gradients are averaged, not
summed.  Alg. 1: the accumulator receives (1/k) of each parameter gradient,
and every k-th backward step the parameters are updated and the accumulator
is reset to zero.

Update rule per tensor p with accumulated gradient D (buffer starts at 0, no
dampening):
    g   = D + wd * p
    buf = mu * buf + g
    p  -= lr * (g + mu * buf)    (Nesterov)      or   p -= lr * buf   (heavy ball)
"""
from __future__ import annotations

import numpy as np


def step(p: np.ndarray, accum: np.ndarray, buf: np.ndarray, lr: float, mu: float,
         wd: float, nesterov: bool):
    """Returns (new_p, new_buf).  The caller zeroes the accumulator."""
    g = accum + wd * p
    nb = mu * buf + g
    if nesterov:
        return p - lr * (g + mu * nb), nb
    return p - lr * nb, nb
