"""2-D convolution (cross-correlation, no bias) on NHWC tensors, KRSC weights.

The forward is the plain definition
    y[n,p,q,o] = sum_{r,s,i} x[n, p*st + r - pad, q*st + s - pad, i] * W[o,r,s,i]
(zero outside the image), evaluated as im2col followed by one matrix product.
The input gradient is the adjoint of that map (col2im scatter-add) and the
weight gradient is the product of the output gradient with the im2col matrix.
The paper computes these through PyTorch's vector-Jacobian products
(Sec. 4.2, "A note on the implementation").
"""
from __future__ import annotations

import numpy as np


def out_size(h: int, r: int, stride: int, pad: int) -> int:
    return (h + 2 * pad - r) // stride + 1


def im2col(x: np.ndarray, r: int, s: int, stride: int, pad: int) -> np.ndarray:
    """[N,H,W,C] -> [N*P*Q, R*S*C] with column index (r, s, c)."""
    n, h, w, c = x.shape
    p, q = out_size(h, r, stride, pad), out_size(w, s, stride, pad)
    xp = np.pad(x, ((0, 0), (pad, pad), (pad, pad), (0, 0)))
    cols = np.empty((n, p, q, r, s, c), dtype=x.dtype)
    for i in range(r):
        for j in range(s):
            cols[:, :, :, i, j, :] = xp[:, i:i + stride * p:stride, j:j + stride * q:stride, :]
    return cols.reshape(n * p * q, r * s * c)


def col2im(cols: np.ndarray, x_shape, r: int, s: int, stride: int, pad: int) -> np.ndarray:
    """Adjoint of im2col: scatter-add columns back into an [N,H,W,C] tensor."""
    n, h, w, c = x_shape
    p, q = out_size(h, r, stride, pad), out_size(w, s, stride, pad)
    cols = cols.reshape(n, p, q, r, s, c)
    xp = np.zeros((n, h + 2 * pad, w + 2 * pad, c), dtype=cols.dtype)
    for i in range(r):
        for j in range(s):
            xp[:, i:i + stride * p:stride, j:j + stride * q:stride, :] += cols[:, :, :, i, j, :]
    return xp[:, pad:pad + h, pad:pad + w, :]


def forward(x: np.ndarray, wt: np.ndarray, stride: int = 1, pad: int | None = None) -> np.ndarray:
    o, r, s, c = wt.shape
    assert x.shape[-1] == c, (x.shape, wt.shape)
    if pad is None:
        pad = (r - 1) // 2
    n, h, w, _ = x.shape
    p, q = out_size(h, r, stride, pad), out_size(w, s, stride, pad)
    y = im2col(x, r, s, stride, pad) @ wt.reshape(o, r * s * c).T
    return y.reshape(n, p, q, o)


def dgrad(dy: np.ndarray, wt: np.ndarray, x_shape, stride: int = 1, pad: int | None = None) -> np.ndarray:
    o, r, s, c = wt.shape
    if pad is None:
        pad = (r - 1) // 2
    dcols = dy.reshape(-1, o) @ wt.reshape(o, r * s * c)
    return col2im(dcols, x_shape, r, s, stride, pad)


def wgrad(x: np.ndarray, dy: np.ndarray, w_shape, stride: int = 1, pad: int | None = None) -> np.ndarray:
    o, r, s, c = w_shape
    if pad is None:
        pad = (r - 1) // 2
    dw = dy.reshape(-1, o).T @ im2col(x, r, s, stride, pad)
    return dw.reshape(o, r, s, c)
