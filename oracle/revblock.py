"""Residual functions and the reversible block (Sec. 3.2, Fig. 2; Eqs. 4-5).

A residual function is a chain of conv -> BN(train) layers with a ReLU after
every BN except the last:
  basic      : conv3x3 - BN - ReLU - conv3x3 - BN
  bottleneck : conv1x1 - BN - ReLU - conv3x3 - BN - ReLU - conv1x1 - BN
It has no skip connection of its own: the skip lives in the coupling.

The activation is split along channels into two equal streams {x1, x2}
(Sec. 3.2 and the caption of Fig. 2).  The primitive is the additive
half-coupling (a, b) -> (a + Phi(b), b), whose inverse subtracts Phi(b)
instead of adding it (Sec. 3.2, "reverse forward").  A block is two
half-couplings, F on x2 then G on the updated first stream:
    y1 = x1 + F(x2)          x2~ = y2 - G(y1)
    y2 = x2 + G(y1)          x1~ = y1 - F(x2~)
(reading: the two-function coupling of the RevNet the paper builds on; the
single-function form of Sec. 3.2 is one half-coupling.)

Storage precision.  `store` maps a tensor to the values a lower-precision
storage format would hold (identity by default, i.e. plain fp64).  It is
applied exactly where the method materialises a tensor: each conv output h
(BN statistics are taken of the stored h), each ReLU activation that feeds the
next conv, the coupling outputs (y, the reconstructed x, the input gradients),
and the gradient tensors dz (masked) and dh (BN input gradient).  The
arithmetic between those points stays fp64, so every ReLU decision is taken on
the stored values.

Backward of a block (Eq. 4 and Eq. 5, Alg. 1 "reconstruct and keep the
computational graph"): the graph of each function is rebuilt while its input
is reconstructed, and the VJP runs through that rebuilt graph, so no separate
forward pass is needed (Sec. 4.2).
"""
from __future__ import annotations

from typing import List, Sequence, Tuple

import numpy as np

from . import bn, conv

Layer = Tuple[np.ndarray, np.ndarray, np.ndarray]   # (W [O,R,S,I], gamma [O], beta [O])


def _identity(a):
    return a


def function_forward(u: np.ndarray, layers: Sequence[Layer], eps: float, store=_identity):
    """Returns (output, graph); graph keeps what the VJP needs."""
    graph = []
    a = u
    for l, (w, g, b) in enumerate(layers):
        h = store(conv.forward(a, w))
        o, cache = bn.forward(h, g, b, eps)
        graph.append((a, h, o, cache))
        a = o if l == len(layers) - 1 else store(np.maximum(o, 0.0))
    return a, graph


def function_vjp(d: np.ndarray, layers: Sequence[Layer], graph, store=_identity):
    """VJP through a rebuilt graph.  Returns (d_input, [(dW, dgamma, dbeta)...]);
    d_input is the unrounded fp64 result (the caller adds and stores it)."""
    grads: List = [None] * len(layers)
    for l in reversed(range(len(layers))):
        w, g, _ = layers[l]
        a, _, o, cache = graph[l]
        if l != len(layers) - 1:
            d = store(d * (o > 0.0))          # ReLU; derivative taken as 0 at 0
        dh, dg, db = bn.backward(d, cache, g)
        dh = store(dh)
        grads[l] = (conv.wgrad(a, dh, w.shape), dg, db)
        d = conv.dgrad(dh, w, a.shape)
    return d, grads


def batch_stats(graph):
    """(mean, var, m) of every BN of a rebuilt graph, for the running statistics."""
    out = []
    for (_, h, _, cache) in graph:
        m = h.shape[0] * h.shape[1] * h.shape[2]
        out.append((cache, m))
    return out


def couple(a: np.ndarray, b: np.ndarray, layers: Sequence[Layer], eps: float,
           store=_identity) -> np.ndarray:
    """Additive half-coupling: a + Phi(b)."""
    f, _ = function_forward(b, layers, eps, store)
    return store(a + f)


def block_forward(x1, x2, f_layers, g_layers, eps, store=_identity):
    """y1 = x1 + F(x2); y2 = x2 + G(y1)."""
    y1 = couple(x1, x2, f_layers, eps, store)
    y2 = couple(x2, y1, g_layers, eps, store)
    return y1, y2


def block_inverse(y1, y2, f_layers, g_layers, eps, store=_identity):
    """Reconstruction only: x2 = y2 - G(y1); x1 = y1 - F(x2)."""
    g, _ = function_forward(y1, g_layers, eps, store)
    x2 = store(y2 - g)
    f, _ = function_forward(x2, f_layers, eps, store)
    return store(y1 - f), x2


def block_reconstruct_vjp(y1, y2, g1, g2, f_layers, g_layers, eps, store=_identity):
    """Reconstruct the block input from its output and take the VJP.

    g1, g2 are the gradients with respect to y1, y2.  Returns a dict with the
    reconstructed inputs x1, x2, the input gradients dx1, dx2, the parameter
    gradients of F and G, and the BN statistics observed while rebuilding.
    """
    gout, g_graph = function_forward(y1, g_layers, eps, store)
    x2 = store(y2 - gout)
    u, dG = function_vjp(g2, g_layers, g_graph, store)
    z1 = store(g1 + u)                # total gradient reaching y1
    fout, f_graph = function_forward(x2, f_layers, eps, store)
    x1 = store(y1 - fout)
    w, dF = function_vjp(z1, f_layers, f_graph, store)
    return dict(x1=x1, x2=x2, dx1=z1, dx2=store(g2 + w), dF=dF, dG=dG,
                stats_F=batch_stats(f_graph), stats_G=batch_stats(g_graph))


def block_vjp(x1, x2, g1, g2, f_layers, g_layers, eps, store=_identity):
    """Plain backpropagation through a block whose input (x1, x2) was kept: the
    forward graph is built from the stored input (no reconstruction) and the
    VJP runs through it.  Same result layout as block_reconstruct_vjp, with
    x1, x2 the given inputs (the input-buffer variant of Table 4)."""
    fout, f_graph = function_forward(x2, f_layers, eps, store)
    y1 = store(x1 + fout)
    _, g_graph = function_forward(y1, g_layers, eps, store)
    u, dG = function_vjp(g2, g_layers, g_graph, store)
    z1 = store(g1 + u)                # total gradient reaching y1
    w, dF = function_vjp(z1, f_layers, f_graph, store)
    return dict(x1=x1, x2=x2, dx1=z1, dx2=store(g2 + w), dF=dF, dG=dG,
                stats_F=batch_stats(f_graph), stats_G=batch_stats(g_graph))
