"""Pins of the optimizer and of gradient accumulation (Sec. 4.1, Alg. 1)."""
import numpy as np
import pytest
import torch

import synth
from oracle import sgd
from oracle.stage import StageState


@pytest.mark.parametrize("nesterov", [True, False])
def test_first_and_second_step_closed_form(nesterov):
    rng = np.random.default_rng(1)
    p = rng.standard_normal(7)
    g1, g2 = rng.standard_normal(7), rng.standard_normal(7)
    lr, mu = 0.1, 0.9
    p1, b1 = sgd.step(p, g1, np.zeros(7), lr, mu, 0.0, nesterov)
    want1 = p - lr * (1 + mu) * g1 if nesterov else p - lr * g1
    np.testing.assert_allclose(p1, want1, rtol=1e-15, atol=1e-15)
    p2, _ = sgd.step(p1, g2, b1, lr, mu, 0.0, nesterov)
    # buf2 = mu g1 + g2
    want2 = p1 - lr * (g2 + mu * (mu * g1 + g2)) if nesterov else p1 - lr * (mu * g1 + g2)
    np.testing.assert_allclose(p2, want2, rtol=1e-14, atol=1e-15)


@pytest.mark.parametrize("nesterov", [True, False])
def test_matches_torch_sgd_with_masked_weight_decay(nesterov):
    rng = np.random.default_rng(4)
    w = rng.standard_normal((3, 4))
    gam = rng.standard_normal(4)
    tw = torch.tensor(w, requires_grad=True)
    tg = torch.tensor(gam, requires_grad=True)
    opt = torch.optim.SGD([{"params": [tw], "weight_decay": 5e-4},
                           {"params": [tg], "weight_decay": 0.0}],
                          lr=0.1, momentum=0.9, nesterov=nesterov)
    bw, bg = np.zeros_like(w), np.zeros_like(gam)
    for it in range(4):
        gw, gg = rng.standard_normal(w.shape), rng.standard_normal(gam.shape)
        tw.grad = torch.tensor(gw)
        tg.grad = torch.tensor(gg)
        opt.step()
        w, bw = sgd.step(w, gw, bw, 0.1, 0.9, 5e-4, nesterov)
        gam, bg = sgd.step(gam, gg, bg, 0.1, 0.9, 0.0, nesterov)
    np.testing.assert_allclose(w, tw.detach().numpy(), rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(gam, tg.detach().numpy(), rtol=1e-13, atol=1e-15)


def _state():
    wl = synth.StageWorkload("t", "fp32", 2, 4, 4, 3, "basic", 1)
    params = [p.astype(np.float64) for p in synth.stage_params(wl, "random")]
    return wl, StageState(params, [n for n, _ in wl.param_shapes()], 2)


def test_accumulation_averages_k_equal_gradients():
    # P7: k backward steps with the same gradient g produce one update with g
    # (averaging, not summing), and no update before the k-th.
    wl, st = _state()
    _, ref = _state()
    rng = np.random.default_rng(0)
    shp = (wl.n, wl.h, wl.w, wl.c_half)
    x1, x2, d1, d2 = [rng.standard_normal(shp) for _ in range(4)]
    y1, y2 = st.forward(x1, x2)
    k = 4
    p0 = [p.copy() for p in st.params]
    for i in range(k):
        # lr=0 until the last step keeps theta (hence g) fixed; accumulation only
        _, _, _, _, g = st.backward(y1, y2, d1, d2, k=k)
        fired = st.update(0.1, 0.9, 0.0, True, k=k)
        assert fired == (i == k - 1)
        if i < k - 1:
            assert all(np.array_equal(a, b) for a, b in zip(st.params, p0))
    ref.backward(y1, y2, d1, d2, k=1)
    ref.update(0.1, 0.9, 0.0, True, k=1)
    for a, b in zip(st.params, ref.params):
        np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-15)
    assert all(np.abs(a).max() == 0 for a in st.accum)


def test_zero_lr_step_is_exact_backprop_of_the_backward_batch():
    # Eq. (5) with an unchanged theta: the step's backward is ordinary backprop
    # of its micro-batch and the forward is the plain stage forward.
    wl, st = _state()
    rng = np.random.default_rng(6)
    shp = (wl.n, wl.h, wl.w, wl.c_half)
    xa1, xa2, xb1, xb2, d1, d2 = [rng.standard_normal(shp) for _ in range(6)]
    yb1, yb2 = st.forward(xb1, xb2)
    fy1, fy2 = st.forward(xa1, xa2)
    out = st.step(xa1, xa2, yb1, yb2, d1, d2, lr=0.0, mu=0.9, wd=0.0)
    np.testing.assert_array_equal(out[0], fy1)
    np.testing.assert_array_equal(out[1], fy2)
    assert np.abs(out[2] - xb1).max() < 1e-12 and np.abs(out[3] - xb2).max() < 1e-12
