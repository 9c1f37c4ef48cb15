"""Pins of the multi-stage schedule (Alg. 1, Eq. 5, App. B delays)."""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

import synth
from oracle.net import PetraNet, head_loss, head_vjp
from tests.torch_ref import revnet

TINY = synth.REVNET18_SCHEDULE.with_(n=4, h=8, w=8, widths=(8, 16, 32, 64), blocks_per_stage=1)


def build(wl, **kw):
    names = [n for n, _ in synth.net_param_shapes(wl)]
    params = [p.astype(np.float64) for p in synth.net_params(wl)]
    # non-trivial BN affine parameters so their gradients are exercised
    rng = np.random.default_rng(12)
    for i, nm in enumerate(names):
        if nm.endswith("gamma"):
            params[i] = 0.5 + rng.random(params[i].shape)
        elif nm.endswith("beta") or nm.endswith("bias"):
            params[i] = 0.2 * rng.standard_normal(params[i].shape)
    return names, params, PetraNet(params, names, len(wl.widths), wl.blocks_per_stage, **kw)


def data(wl, count):
    rng = np.random.default_rng(21)
    imgs = rng.standard_normal((count, wl.n, wl.h, wl.w, wl.c_img))
    labs = rng.integers(0, wl.classes, size=(count, wl.n))
    return imgs, labs


def test_head_matches_torch():
    rng = np.random.default_rng(0)
    x = rng.standard_normal((5, 3, 2, 8))
    w = rng.standard_normal((4, 8))
    b = rng.standard_normal(4)
    lab = rng.integers(0, 4, 5)
    loss, cache = head_loss(x, w, b, lab)
    xt = torch.tensor(x, requires_grad=True)
    wt = torch.tensor(w, requires_grad=True)
    bt = torch.tensor(b, requires_grad=True)
    lt = Fn.cross_entropy(xt.mean(dim=(1, 2)) @ wt.T + bt, torch.tensor(lab))
    lt.backward()
    assert abs(loss - lt.item()) < 1e-12
    dx, dw, db = head_vjp(w, lab, cache)
    np.testing.assert_allclose(dx, xt.grad.numpy(), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(dw, wt.grad.numpy(), rtol=1e-12, atol=1e-15)
    np.testing.assert_allclose(db, bt.grad.numpy(), rtol=1e-12, atol=1e-15)


def test_tick_table_and_delays():
    names, params, net = build(TINY)
    imgs, labs = data(TINY, 3)
    J = 4
    T = 3 + 2 * J
    for t in range(T):
        net.tick(t, lambda m: imgs[m], lambda m: labs[m], 3, 0.0, 0.9, 0.0)
    fwd_at, bwd_at = {}, {}
    for (t, j, m, mb) in net.trace:
        if m is not None:
            fwd_at[(j, m)] = t
        if mb is not None:
            bwd_at[(j, mb)] = t
    for j in range(J):
        for m in range(3):
            assert fwd_at[(j, m)] == m + j                 # one hop per tick forward
            assert bwd_at[(j, m)] - fwd_at[(j, m)] == 2 * (J - 1 - j)   # tau = 2(J - j), 1-based j
    # every micro-batch went through every stage forward and backward once
    assert len(fwd_at) == len(bwd_at) == 3 * J
    assert all(not st.buffer for st in net.stages)       # buffers drained


def test_zero_lr_gives_exact_backprop_per_microbatch():
    # P8: with theta frozen, the schedule's accumulated gradients equal the sum
    # of end-to-end backprop gradients of the micro-batches.
    names, params, net = build(TINY)
    imgs, labs = data(TINY, 3)
    K = 1000          # never reaches an update; the accumulator holds sum / K
    for t in range(3 + 2 * 4):
        net.tick(t, lambda m: imgs[m], lambda m: labs[m], 3, 0.0, 0.9, 0.0, k=K)
    leaves = [torch.tensor(p, requires_grad=True) for p in params]
    total = 0
    for m in range(3):
        logits = revnet(imgs[m], leaves, names, 4, 1)
        total = total + Fn.cross_entropy(logits, torch.tensor(labs[m]).long())
    total.backward()
    got = {}
    for st in net.stages:
        for nm, a in zip(st.names, st.accum):
            got[nm] = a * K
    for nm, leaf in zip(names, leaves):
        ref = leaf.grad.numpy()
        # some gradients vanish identically (a last-BN beta feeding a BN'd
        # downsampling sees a shift-invariant loss): absolute floor 1e-12
        err = np.linalg.norm(got[nm] - ref)
        assert err <= 1e-9 * np.linalg.norm(ref) + 1e-12, (nm, err)


def test_single_stage_is_plain_sgd():
    # P8: J = 1 has no delay: forward, loss, backward and update each tick.
    wl = TINY.with_(widths=(8,))
    names, params, net = build(wl)
    imgs, labs = data(wl, 2)
    leaves = [torch.tensor(p, requires_grad=True) for p in params]
    groups = [{"params": [l], "weight_decay": 5e-4 if nm.endswith("weight") else 0.0}
              for nm, l in zip(names, leaves)]
    opt = torch.optim.SGD(groups, lr=0.1, momentum=0.9, nesterov=True)
    for t in range(3):
        loss = net.tick(t, lambda m: imgs[m % 2], lambda m: labs[m % 2], 3, 0.1, 0.9, 5e-4)
        opt.zero_grad()
        lt = Fn.cross_entropy(revnet(imgs[t % 2], leaves, names, 1, 1), torch.tensor(labs[t % 2]).long())
        assert abs(loss - lt.item()) < 1e-10
        lt.backward()
        opt.step()
    for nm, p, leaf in zip(names, net.stages[0].params, leaves):
        np.testing.assert_allclose(p, leaf.detach().numpy(), rtol=1e-9, atol=1e-12, err_msg=nm)


def test_backprop_step_is_sgd_on_end_to_end_gradients():
    # The sequential baseline of the iteration-time comparison (Table 5): with
    # J = 4 stages and blocks rebuilt from their outputs it is plain SGD on the
    # end-to-end gradient, step after step (autograd over the non-reversible
    # network as the independent reference).
    names, params, net = build(TINY)
    imgs, labs = data(TINY, 2)
    leaves = [torch.tensor(p, requires_grad=True) for p in params]
    groups = [{"params": [l], "weight_decay": 5e-4 if nm.endswith("weight") else 0.0}
              for nm, l in zip(names, leaves)]
    opt = torch.optim.SGD(groups, lr=0.05, momentum=0.9, nesterov=True)
    for t in range(3):
        loss = net.backprop_step(imgs[t % 2], labs[t % 2], 0.05, 0.9, 5e-4)
        opt.zero_grad()
        lt = Fn.cross_entropy(revnet(imgs[t % 2], leaves, names, 4, 1),
                              torch.tensor(labs[t % 2]).long())
        assert abs(loss - lt.item()) < 1e-10
        lt.backward()
        opt.step()
    got = {nm: p for st in net.stages for nm, p in zip(st.names, st.params)}
    for nm, leaf in zip(names, leaves):
        np.testing.assert_allclose(got[nm], leaf.detach().numpy(), rtol=1e-9, atol=1e-12,
                                   err_msg=nm)


def test_backprop_step_with_accumulation_updates_every_k():
    # k = 2: the first step only accumulates; the second applies the mean of
    # the two end-to-end gradients (Sec. 4.1, gradient accumulation).
    names, params, net = build(TINY)
    imgs, labs = data(TINY, 2)
    net.backprop_step(imgs[0], labs[0], 0.05, 0.0, 0.0, k=2)
    p1 = {nm: p.copy() for st in net.stages for nm, p in zip(st.names, st.params)}
    for nm, p in zip(names, params):
        np.testing.assert_array_equal(p1[nm], p)
    net.backprop_step(imgs[1], labs[1], 0.05, 0.0, 0.0, k=2)
    leaves = [torch.tensor(p, requires_grad=True) for p in params]
    total = sum(Fn.cross_entropy(revnet(imgs[m], leaves, names, 4, 1), torch.tensor(labs[m]).long())
                for m in range(2)) / 2
    total.backward()
    got = {nm: p for st in net.stages for nm, p in zip(st.names, st.params)}
    for nm, p, leaf in zip(names, params, leaves):
        want = p - 0.05 * leaf.grad.numpy()
        np.testing.assert_allclose(got[nm], want, rtol=1e-9, atol=1e-12, err_msg=nm)
