"""Pins of the multi-stage schedule (Alg. 1, Eq. 5, App. B delays)."""
import copy

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


def _stage_vjp_torch(names, j, blocks, P, x_in, u, g):
    """VJP of stage j in torch autograd (fp64): front layer at its buffered input
    x_in, blocks at the block input u, parameters P (by name), cotangent g on
    the block output; returns the parameter gradients by name."""
    from tests.torch_ref import front, nchw, stage_blocks
    leaves = {nm: torch.tensor(P[nm], requires_grad=True) for nm in names}
    xi = nchw(x_in[0]) if x_in[1] is None else torch.cat([nchw(x_in[0]), nchw(x_in[1])], 1)
    u1 = nchw(u[0]).clone().requires_grad_(True)
    u2 = nchw(u[1]).clone().requires_grad_(True)
    y1, y2 = stage_blocks(u1, u2, leaves, j, blocks)
    ((y1 * nchw(g[0])).sum() + (y2 * nchw(g[1])).sum()).backward()
    du = torch.cat([u1.grad, u2.grad], 1)
    (front(xi, leaves, j) * du).sum().backward()
    return {nm: leaves[nm].grad.numpy() for nm in names}


@pytest.mark.parametrize("use_inputs,use_params", [(False, False), (True, False), (False, True),
                                                   (True, True)])
def test_buffer_variants_take_the_vjp_at_their_definition(use_inputs, use_params):
    # Table 4 variants: every recorded backward is the VJP of its stage at the
    # block input and parameters its variant prescribes, with the received
    # cotangent; the block input is the stored one (input buffer) or the
    # inverse of the received output under the latest parameters; the
    # parameters are the forward's (parameter buffer) or the latest.
    names, params, net = build(TINY)
    net.use_inputs, net.use_params = use_inputs, use_params
    net.record = {}
    imgs, labs = data(TINY, 3)
    J = 4
    latest, at_fwd = {}, {}
    for t in range(3 + 2 * J):
        for j, st in enumerate(net.stages):
            for m, P in st.stash.items():
                at_fwd.setdefault((j, m), dict(zip(st.names, P)))
            latest[(j, t)] = dict(zip(st.names, [p.copy() for p in st.params]))
        net.tick(t, lambda m: imgs[m], lambda m: labs[m], 3, 0.05, 0.9, 5e-4)
    from oracle import revblock
    stale = 0
    for (j, m), r in net.record.items():
        if j == J - 1:
            continue    # forward and backward in one tick: nothing is delayed
        st = net.stages[j]
        t_b = m + 2 * J - 2 - j
        want_P = at_fwd[(j, m)] if use_params else latest[(j, t_b)]
        for nm, p in zip(st.names, r["P"]):
            np.testing.assert_array_equal(p, want_P[nm])
        stale += any(np.abs(latest[(j, t_b)][nm] - at_fwd[(j, m)][nm]).max() > 0
                     for nm in st.names)
        u1, u2 = r["u"]
        if use_inputs:
            # the forward's block input: front layer at the forward's parameters
            from tests.torch_ref import front, nchw
            Pf = {nm: torch.tensor(v) for nm, v in at_fwd[(j, m)].items()}
            x = r["x_in"]
            xi = nchw(x[0]) if x[1] is None else torch.cat([nchw(x[0]), nchw(x[1])], 1)
            a = front(xi, Pf, j).permute(0, 2, 3, 1).numpy()
            c = a.shape[-1] // 2
            np.testing.assert_allclose(u1, a[..., :c], rtol=1e-10, atol=1e-12)
            np.testing.assert_allclose(u2, a[..., c:], rtol=1e-10, atol=1e-12)
        else:
            # reconstruction under the latest parameters maps back onto the received output
            v1, v2 = u1, u2
            for b in range(TINY.blocks_per_stage):
                v1, v2 = revblock.block_forward(v1, v2, st._layers(b, 0, r["P"] if not use_params
                                                                  else [latest[(j, t_b)][nm] for nm in st.names]),
                                                st._layers(b, 1, r["P"] if not use_params
                                                           else [latest[(j, t_b)][nm] for nm in st.names]),
                                                st.eps)
            np.testing.assert_allclose(v1, r["y"][0], rtol=1e-9, atol=1e-10)
            np.testing.assert_allclose(v2, r["y"][1], rtol=1e-9, atol=1e-10)
        tg = _stage_vjp_torch(st.names, j, TINY.blocks_per_stage, dict(zip(st.names, r["P"])),
                              r["x_in"], r["u"], r["g"])
        for nm, gv in zip(st.names, r["grads"]):
            err = np.linalg.norm(gv - tg[nm])
            assert err <= 1e-9 * np.linalg.norm(tg[nm]) + 1e-12, (j, m, nm, err)
    assert stale >= 3   # backwards whose stage was updated after their forward


def test_both_buffers_give_exact_delayed_gradients():
    # Input and parameter buffers together (PipeDream weight stashing): the
    # gradient stage j accumulates for micro-batch m is the end-to-end gradient
    # of m's loss through the network at the parameters each stage's forward
    # of m used (App. B, the standard delayed gradient).
    names, params, net = build(TINY)
    net.use_inputs = net.use_params = True
    net.record = {}
    imgs, labs = data(TINY, 3)
    J = 4
    at_fwd = {}
    for t in range(3 + 2 * J):
        net.tick(t, lambda m: imgs[m], lambda m: labs[m], 3, 0.05, 0.9, 5e-4)
        for j, st in enumerate(net.stages):
            for m, P in st.stash.items():
                at_fwd.setdefault((j, m), dict(zip(st.names, P)))
    for m in range(3):
        # the last stage stashes and consumes within one tick: its forward used the
        # parameters it had before that tick's update, as the record shows
        P = {}
        for j, st in enumerate(net.stages):
            P.update(at_fwd[(j, m)] if (j, m) in at_fwd else
                     dict(zip(st.names, net.record[(j, m)]["P"])))
        leaves = [torch.tensor(P[nm], requires_grad=True) for nm in names]
        loss = Fn.cross_entropy(revnet(imgs[m], leaves, names, J, 1), torch.tensor(labs[m]).long())
        loss.backward()
        for j, st in enumerate(net.stages):
            for nm, gv in zip(st.names, net.record[(j, m)]["grads"]):
                ref = leaves[names.index(nm)].grad.numpy()
                err = np.linalg.norm(gv - ref)
                assert err <= 1e-9 * np.linalg.norm(ref) + 1e-12, (j, m, nm, err)


def test_probes_leave_the_schedule_untouched_and_agree_at_the_last_stage():
    names, params, net = build(TINY)
    imgs, labs = data(TINY, 8)
    J = 4
    for t in range(2 * J):
        net.tick(t, lambda m: imgs[m], lambda m: labs[m], 8, 0.05, 0.9, 5e-4)
    before = copy.deepcopy(net)
    t = 2 * J
    probes = {mode: net.probe_tick(t, lambda m: imgs[m], lambda m: labs[m], 8, *mode)
              for mode in [(False, False), (True, True)]}
    m_last = t - (J - 1)
    e2e = net.probe_backprop(imgs[m_last], labs[m_last])
    for a, b in zip(before.stages, net.stages):
        for p, q in zip(a.params, b.params):
            np.testing.assert_array_equal(p, q)
        assert a.stash.keys() == b.stash.keys() and a.inbuf.keys() == b.inbuf.keys()
    last = net.stages[-1].names
    for nm in last:
        # no delay at the last stage: the PETRA and delayed gradients coincide
        a, b = probes[(False, False)][nm], probes[(True, True)][nm]
        assert np.linalg.norm(a - b) <= 1e-9 * np.linalg.norm(b) + 1e-12, nm
    # the end-to-end probe is autograd's gradient at the current parameters
    cur = {nm: p for st in net.stages for nm, p in zip(st.names, st.params)}
    leaves = [torch.tensor(cur[nm], requires_grad=True) for nm in names]
    Fn.cross_entropy(revnet(imgs[m_last], leaves, names, J, 1),
                     torch.tensor(labs[m_last]).long()).backward()
    for nm, leaf in zip(names, leaves):
        ref = leaf.grad.numpy()
        assert np.linalg.norm(e2e[nm] - ref) <= 1e-9 * np.linalg.norm(ref) + 1e-12, nm
    # stage 0 has a delay of 2(J-1) ticks with updates in between: the variants differ
    s0 = net.stages[0].names
    assert max(np.abs(probes[(False, False)][nm] - probes[(True, True)][nm]).max() for nm in s0) > 0


def test_split_fronts_tick_table_and_exact_backprop_when_frozen():
    # Paper-style split (each stem/downsampling and each block its own stage):
    # J = 8 for 4 levels of one block; delays 2(J-1-j); with theta
    # frozen the accumulated gradients are exact backprop even though the
    # reversible stages rebuild their inputs from the reconstructions sent by
    # the stage above (Eq. 4).
    names, params, _ = build(TINY)
    net = PetraNet(params, names, 4, 1, split_fronts=True)
    assert net.J == 8
    assert [st.front for st in net.stages] == ["stem", None, "trans", None, "trans", None, "trans", None]
    assert [st.blocks for st in net.stages] == [0, 1, 0, 1, 0, 1, 0, 1]
    imgs, labs = data(TINY, 3)
    J = net.J
    K = 1000
    for t in range(3 + 2 * J):
        net.tick(t, lambda m: imgs[m], lambda m: labs[m], 3, 0.0, 0.9, 0.0, k=K)
    fwd_at, bwd_at = {}, {}
    for (t, j, m, mb) in net.trace:
        if m is not None:
            fwd_at[(j, m)] = t
        if mb is not None:
            bwd_at[(j, mb)] = t
    for j in range(J):
        for m in range(3):
            assert bwd_at[(j, m)] - fwd_at[(j, m)] == 2 * (J - 1 - j)
    assert all(not st.buffer for st in net.stages)
    leaves = [torch.tensor(p, requires_grad=True) for p in params]
    total = 0
    for m in range(3):
        total = total + Fn.cross_entropy(revnet(imgs[m], leaves, names, 4, 1),
                                         torch.tensor(labs[m]).long())
    total.backward()
    got = {nm: a * K for st in net.stages for nm, a in zip(st.names, st.accum)}
    assert set(got) == set(names)
    for nm, leaf in zip(names, leaves):
        ref = leaf.grad.numpy()
        err = np.linalg.norm(got[nm] - ref)
        assert err <= 1e-9 * np.linalg.norm(ref) + 1e-12, (nm, err)


def test_split_fronts_reversible_stage_reconstructs_from_received_reconstruction():
    # Two blocks per level, each its own stage (J = 12): with updates between
    # forward and backward, a reversible stage's block input is the inverse,
    # under its current parameters, of what the stage above sent back, and when
    # that stage is reversible too, what it sent is its own reconstruction.
    wl = TINY.with_(blocks_per_stage=2)
    names, params, _ = build(wl)
    net = PetraNet(params, names, 4, 2, split_fronts=True)
    assert net.J == 12
    net.record = {}
    imgs, labs = data(wl, 4)
    for t in range(4 + 2 * net.J):
        net.tick(t, lambda m: imgs[m], lambda m: labs[m], 4, 0.05, 0.9, 5e-4)
    from oracle import revblock
    checked = chained = 0
    for (j, m), r in net.record.items():
        st = net.stages[j]
        if st.front or st.last:
            continue
        above = net.stages[j + 1]
        if above.front is None and (j + 1, m) in net.record:
            # the stage above is reversible: it sent back the input it used
            np.testing.assert_array_equal(r["y"][0], net.record[(j + 1, m)]["u"][0])
            np.testing.assert_array_equal(r["y"][1], net.record[(j + 1, m)]["u"][1])
            chained += 1
        # forward of the used input under the parameters of the backward gives
        # back the received output
        v1, v2 = r["u"]
        P = r["P"]
        for b in range(st.blocks):
            v1, v2 = revblock.block_forward(v1, v2, st._layers(b, 0, P), st._layers(b, 1, P), st.eps)
        np.testing.assert_allclose(v1, r["y"][0], rtol=1e-9, atol=1e-10)
        np.testing.assert_allclose(v2, r["y"][1], rtol=1e-9, atol=1e-10)
        checked += 1
    assert checked >= 12 and chained >= 4
