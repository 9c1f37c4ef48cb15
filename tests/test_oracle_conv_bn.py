"""Pins of the oracle's conv and BN primitives against torch CPU (fp64) and a
brute-force loop over the definition."""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

from oracle import bn, conv
from tests.torch_ref import nchw, nhwc, oihw

CASES = [  # (N, H, W, C_in, C_out, R, stride)
    (2, 5, 6, 3, 4, 3, 1),
    (2, 4, 4, 8, 5, 1, 1),
    (3, 6, 6, 4, 7, 1, 2),
    (1, 7, 5, 3, 8, 3, 1),
]


@pytest.mark.parametrize("case", CASES)
def test_conv_matches_torch(case):
    n, h, w, ci, co, r, st = case
    rng = np.random.default_rng(7)
    x = rng.standard_normal((n, h, w, ci))
    wt = rng.standard_normal((co, r, r, ci))
    pad = (r - 1) // 2
    y = conv.forward(x, wt, stride=st, pad=pad)
    xt = nchw(x).clone().requires_grad_(True)
    wtt = oihw(wt).clone().requires_grad_(True)
    yt = Fn.conv2d(xt, wtt, stride=st, padding=pad)
    np.testing.assert_allclose(y, nhwc(yt).detach().numpy(), rtol=1e-12, atol=1e-12)
    dy = rng.standard_normal(y.shape)
    (yt * nchw(dy)).sum().backward()
    dx = conv.dgrad(dy, wt, x.shape, stride=st, pad=pad)
    dw = conv.wgrad(x, dy, wt.shape, stride=st, pad=pad)
    np.testing.assert_allclose(dx, nhwc(xt.grad).numpy(), rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(dw, wtt.grad.permute(0, 2, 3, 1).numpy(), rtol=1e-11, atol=1e-11)


def test_conv_bruteforce_definition():
    rng = np.random.default_rng(3)
    n, h, w, ci, co = 2, 4, 3, 2, 3
    x = rng.standard_normal((n, h, w, ci))
    wt = rng.standard_normal((co, 3, 3, ci))
    y = conv.forward(x, wt)
    ref = np.zeros((n, h, w, co))
    for a in range(n):
        for p in range(h):
            for q in range(w):
                for o in range(co):
                    acc = 0.0
                    for r in range(3):
                        for s in range(3):
                            ih, iw = p + r - 1, q + s - 1
                            if 0 <= ih < h and 0 <= iw < w:
                                for i in range(ci):
                                    acc += x[a, ih, iw, i] * wt[o, r, s, i]
                    ref[a, p, q, o] = acc
    np.testing.assert_allclose(y, ref, rtol=1e-13, atol=1e-13)


def test_conv_adjoint_identity():
    # <conv(x), dy> == <x, dgrad(dy)> == <W, wgrad(x, dy)>
    rng = np.random.default_rng(5)
    x = rng.standard_normal((2, 5, 5, 3))
    wt = rng.standard_normal((4, 3, 3, 3))
    y = conv.forward(x, wt)
    dy = rng.standard_normal(y.shape)
    lhs = (y * dy).sum()
    assert abs(lhs - (x * conv.dgrad(dy, wt, x.shape)).sum()) < 1e-10
    assert abs(lhs - (wt * conv.wgrad(x, dy, wt.shape)).sum()) < 1e-10


def test_bn_matches_torch_and_invariants():
    rng = np.random.default_rng(11)
    h = rng.standard_normal((4, 3, 5, 6)) * 3 + 1.5
    g = rng.random(6) + 0.5
    b = rng.standard_normal(6)
    eps = 1e-5
    out, cache = bn.forward(h, g, b, eps)
    ht = nchw(h).clone().requires_grad_(True)
    gt = torch.tensor(g, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    rm = torch.zeros(6, dtype=torch.float64)
    rv = torch.ones(6, dtype=torch.float64)
    ot = Fn.batch_norm(ht, rm, rv, gt, bt, training=True, momentum=0.1, eps=eps)
    np.testing.assert_allclose(out, nhwc(ot).detach().numpy(), rtol=1e-12, atol=1e-12)
    d = rng.standard_normal(out.shape)
    (ot * nchw(d)).sum().backward()
    dh, dg, db = bn.backward(d, cache, g)
    np.testing.assert_allclose(dh, nhwc(ht.grad).numpy(), rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(dg, gt.grad.numpy(), rtol=1e-11)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-11)
    # running statistics (unbiased variance, momentum 0.1) equal torch's
    m = 4 * 3 * 5
    nm, nv = bn.running_update(np.zeros(6), np.ones(6), cache, m, 0.1)
    np.testing.assert_allclose(nm, rm.numpy(), rtol=1e-12)
    np.testing.assert_allclose(nv, rv.numpy(), rtol=1e-12)
    # invariants: the BN input gradient is orthogonal to 1 and to xhat
    xhat = cache[0]
    assert np.abs(dh.sum(axis=(0, 1, 2))).max() < 1e-10
    # sum(dh * xhat) vanishes up to the epsilon term: sum(xhat^2) = m var/(var+eps)
    var_b = h.var(axis=(0, 1, 2))
    resid = g * cache[1] * dg * eps / (var_b + eps)
    np.testing.assert_allclose((dh * xhat).sum(axis=(0, 1, 2)), resid, rtol=1e-6, atol=1e-14)
    # output moments: mean beta, variance gamma^2 sigma^2 / (sigma^2 + eps)
    var = h.var(axis=(0, 1, 2))
    np.testing.assert_allclose(out.mean(axis=(0, 1, 2)), b, atol=1e-12)
    np.testing.assert_allclose(out.var(axis=(0, 1, 2)), g * g * var / (var + eps), rtol=1e-10)


def test_bias_before_bn_has_zero_gradient():
    # A per-channel bias added before train-mode BN receives sum(dh) = 0, which
    # is why the convolutions carry no bias.
    rng = np.random.default_rng(2)
    h = rng.standard_normal((3, 4, 4, 5))
    bias = torch.zeros(5, dtype=torch.float64, requires_grad=True)
    ht = nchw(h)
    o = Fn.batch_norm(ht + bias.view(1, 5, 1, 1), None, None, None, None, training=True, eps=1e-5)
    (o * nchw(rng.standard_normal(h.shape))).sum().backward()
    assert bias.grad.abs().max().item() < 1e-12
