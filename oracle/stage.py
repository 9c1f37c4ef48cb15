"""A reversible stage: B blocks in sequence, with its single parameter copy,
gradient accumulator, optimizer state and BN running statistics.

Eq. (5) for an intermediate reversible stage j at time step t:
    forward     x_j      = F_j(x_{j-1}, theta^t)
    reconstruct x~_{j-1} = F_j^{-1}(x~_j, theta^t)
    input grad  delta_j  = d_x F_j(x~_{j-1}, theta^t)^T delta_{j+1}
    param grad  Delta_j  = d_theta F_j(x~_{j-1}, theta^t)^T delta_{j+1}
    update      theta^{t+1} = Optimizer(theta^t, Delta_j)
Both the forward and the backward of a step read the same, current theta^t;
no stashed copy exists (Sec. 3.3).  Alg. 1 accumulates (1/k) of each gradient
and updates every k-th backward step.

Readings: the update counts backward steps from 1 and fires when the count is
a multiple of k; BN running statistics (mean 0, variance 1 at start) move only
in the backward recompute (Sec. 4.1).
"""
from __future__ import annotations

from typing import Callable, List, Optional, Sequence

import numpy as np

from . import bn, revblock, sgd


class StageState:
    """Oracle state of one reversible stage.

    params: list of arrays in canonical order (per block: F then G; per conv:
    weight [O,R,S,I], gamma, beta).  names: their names (used only for the
    weight-decay mask: tensors whose name ends in "weight" are decayed).
    n_convs: convs per residual function (2 basic, 3 bottleneck).
    weight_view: optional map applied to conv weights before use (e.g. the
    rounding of a lower-precision compute copy); defaults to identity.
    store: optional map giving the values a lower-precision storage format
    holds, applied where the method materialises activations and activation
    gradients (see revblock); defaults to identity (plain fp64).
    """

    def __init__(self, params: Sequence[np.ndarray], names: Sequence[str], n_convs: int,
                 eps: float = 1e-5, bn_momentum: float = 0.1, dtype=np.float64,
                 weight_view: Optional[Callable[[np.ndarray], np.ndarray]] = None,
                 store: Optional[Callable[[np.ndarray], np.ndarray]] = None):
        self.dtype = dtype
        self.params = [np.array(p, dtype=dtype) for p in params]
        self.names = list(names)
        self.n_convs = n_convs
        self.eps = eps
        self.bn_momentum = bn_momentum
        self.weight_view = weight_view
        if store is None:
            self.store = lambda a: a
        else:
            self.store = lambda a: np.asarray(store(np.asarray(a, np.float32)), dtype=dtype)
        self.accum = [np.zeros_like(p) for p in self.params]
        self.buf = [np.zeros_like(p) for p in self.params]
        per_fn = 3 * n_convs
        assert len(self.params) % (2 * per_fn) == 0
        self.blocks = len(self.params) // (2 * per_fn)
        # running statistics, one (mean, var) per BN in canonical order
        self.run_mean = [np.zeros(self.params[i + 1].shape, dtype) for i in self._bn_slots()]
        self.run_var = [np.ones(self.params[i + 1].shape, dtype) for i in self._bn_slots()]
        self.t = 0          # backward steps taken since the start

    # -- parameter plumbing ------------------------------------------------
    def _bn_slots(self) -> List[int]:
        """Index of each conv weight (the BN gamma/beta follow it)."""
        return list(range(0, len(self.params), 3))

    def _layers(self, b: int, f: int):
        per_fn = 3 * self.n_convs
        base = (2 * b + f) * per_fn
        out = []
        for l in range(self.n_convs):
            w, g, be = self.params[base + 3 * l: base + 3 * l + 3]
            if self.weight_view is not None:
                w = np.asarray(self.weight_view(w.astype(np.float32)), dtype=self.dtype)
            out.append((w, g, be))
        return out

    # -- Eq. (5), first line ------------------------------------------------
    def forward(self, x1: np.ndarray, x2: np.ndarray):
        x1 = np.asarray(x1, self.dtype)
        x2 = np.asarray(x2, self.dtype)
        for b in range(self.blocks):
            x1, x2 = revblock.block_forward(x1, x2, self._layers(b, 0), self._layers(b, 1), self.eps,
                                            self.store)
        return x1, x2

    def inverse(self, y1: np.ndarray, y2: np.ndarray):
        y1 = np.asarray(y1, self.dtype)
        y2 = np.asarray(y2, self.dtype)
        for b in reversed(range(self.blocks)):
            y1, y2 = revblock.block_inverse(y1, y2, self._layers(b, 0), self._layers(b, 1), self.eps,
                                            self.store)
        return y1, y2

    # -- Eq. (5), lines two to four; Alg. 1 accumulation -----------------------
    def backward(self, y1, y2, dy1, dy2, k: int = 1):
        """Reconstruct the stage input and take the VJP with the current theta.

        Adds (1/k) of the parameter gradient to the accumulator, updates the BN
        running statistics and returns (x1~, x2~, dx1, dx2, grads) where grads
        is the unscaled parameter gradient in canonical order.
        """
        y1 = np.asarray(y1, self.dtype)
        y2 = np.asarray(y2, self.dtype)
        g1 = np.asarray(dy1, self.dtype)
        g2 = np.asarray(dy2, self.dtype)
        grads: List[Optional[np.ndarray]] = [None] * len(self.params)
        per_fn = 3 * self.n_convs
        for b in reversed(range(self.blocks)):
            r = revblock.block_reconstruct_vjp(y1, y2, g1, g2, self._layers(b, 0),
                                               self._layers(b, 1), self.eps, self.store)
            for f, key in ((0, "dF"), (1, "dG")):
                base = (2 * b + f) * per_fn
                stats = r["stats_F" if f == 0 else "stats_G"]
                for l, (dw, dg, db) in enumerate(r[key]):
                    grads[base + 3 * l] = dw
                    grads[base + 3 * l + 1] = dg
                    grads[base + 3 * l + 2] = db
                    slot = (base + 3 * l) // 3
                    cache, m = stats[l]
                    self.run_mean[slot], self.run_var[slot] = bn.running_update(
                        self.run_mean[slot], self.run_var[slot], cache, m, self.bn_momentum)
            y1, y2, g1, g2 = r["x1"], r["x2"], r["dx1"], r["dx2"]
        for a, g in zip(self.accum, grads):
            a += g / k
        self.t += 1
        return y1, y2, g1, g2, grads

    # -- Eq. (5), last line ------------------------------------------------
    def update(self, lr: float, mu: float, wd: float, nesterov: bool = True, k: int = 1) -> bool:
        """Apply the optimizer if the backward count is a multiple of k."""
        if self.t == 0 or self.t % k != 0:
            return False
        for i, name in enumerate(self.names):
            wdp = wd if name.endswith("weight") else 0.0
            self.params[i], self.buf[i] = sgd.step(self.params[i], self.accum[i], self.buf[i],
                                                   lr, mu, wdp, nesterov)
            self.accum[i] = np.zeros_like(self.accum[i])
        return True

    def step(self, x1, x2, y1, y2, dy1, dy2, lr, mu, wd, nesterov=True, k=1):
        """One PETRA stage step: forward of one micro-batch and reconstruct+VJP
        of another, both with theta^t, then the update (Eq. 5)."""
        fy1, fy2 = self.forward(x1, x2)
        out = self.backward(y1, y2, dy1, dy2, k)
        self.update(lr, mu, wd, nesterov, k)
        return (fy1, fy2) + out[:4]
