"""Pins of the oracle's reversible block and stage (Eqs. 2-5)."""
import numpy as np
import pytest
import torch

import synth
from oracle import revblock
from oracle.stage import StageState
from tests.torch_ref import block, nchw, nhwc, oihw, residual_fn


def tiny(kind="basic", blocks=1, n=2, h=4, w=4, c=4, mid=3):
    return synth.StageWorkload("tiny", "fp32", n, h, w, c, kind, blocks, c_mid=mid)


def make_state(wl, affine="random"):
    params = [p.astype(np.float64) for p in synth.stage_params(wl, affine)]
    names = [nm for nm, _ in wl.param_shapes()]
    return StageState(params, names, 2 if wl.kind == "basic" else 3)


def rand_io(wl, seed=0):
    rng = np.random.default_rng(seed)
    shp = (wl.n, wl.h, wl.w, wl.c_half)
    return [rng.standard_normal(shp) for _ in range(4)]


@pytest.mark.parametrize("kind,blocks", [("basic", 1), ("basic", 3), ("bottleneck", 2)])
def test_inverse_of_forward_is_identity(kind, blocks):
    # P1: with theta frozen, F^{-1}(F(x)) == x (Eq. 4)
    wl = tiny(kind, blocks, n=3, h=5, w=4, c=6, mid=4)
    st = make_state(wl)
    x1, x2, _, _ = rand_io(wl)
    y1, y2 = st.forward(x1, x2)
    r1, r2 = st.inverse(y1, y2)
    assert np.abs(r1 - x1).max() < 1e-12 and np.abs(r2 - x2).max() < 1e-12
    # and the backward's reconstruction is the same inverse
    before = [m.copy() for m in st.run_mean]
    rx1, rx2, *_ = st.backward(y1, y2, *rand_io(wl, 1)[:2])
    assert np.abs(rx1 - x1).max() < 1e-12 and np.abs(rx2 - x2).max() < 1e-12
    assert any(np.abs(a - b).max() > 0 for a, b in zip(before, st.run_mean))


def torch_stage_grads(wl, st, x1, x2, dy1, dy2):
    """Ordinary backprop through stored activations (torch autograd, fp64)."""
    ps = [torch.tensor(p, requires_grad=True) for p in st.params]
    t1 = nchw(x1).clone().requires_grad_(True)
    t2 = nchw(x2).clone().requires_grad_(True)
    a1, a2 = t1, t2
    n = st.n_convs
    for b in range(st.blocks):
        def lay(f):
            base = (2 * b + f) * 3 * n
            return [(ps[base + 3 * l].permute(0, 3, 1, 2), ps[base + 3 * l + 1], ps[base + 3 * l + 2])
                    for l in range(n)]
        a1, a2 = block(a1, a2, lay(0), lay(1))
    loss = (a1 * nchw(dy1)).sum() + (a2 * nchw(dy2)).sum()
    loss.backward()
    return (nhwc(a1).detach().numpy(), nhwc(a2).detach().numpy(),
            nhwc(t1.grad).numpy(), nhwc(t2.grad).numpy(), [p.grad.numpy() for p in ps])


@pytest.mark.parametrize("kind,blocks", [("basic", 1), ("basic", 2), ("bottleneck", 2)])
def test_frozen_reconstruct_vjp_equals_backprop(kind, blocks):
    # P2: with theta frozen, the gradients computed from reconstructed inputs
    # equal standard backprop on stored activations (Eqs. 2-4).
    wl = tiny(kind, blocks, n=2, h=5, w=5, c=4, mid=3)
    st = make_state(wl)
    x1, x2, dy1, dy2 = rand_io(wl, 3)
    y1, y2 = st.forward(x1, x2)
    ty1, ty2, tdx1, tdx2, tgrads = torch_stage_grads(wl, st, x1, x2, dy1, dy2)
    np.testing.assert_allclose(y1, ty1, rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(y2, ty2, rtol=1e-11, atol=1e-11)
    rx1, rx2, dx1, dx2, grads = st.backward(y1, y2, dy1, dy2)
    for a, b in ((dx1, tdx1), (dx2, tdx2)):
        assert np.linalg.norm(a - b) <= 1e-10 * np.linalg.norm(b)
    for g, tg in zip(grads, tgrads):
        assert np.linalg.norm(g - tg) <= 1e-10 * max(np.linalg.norm(tg), 1e-30)


def test_finite_differences_tiny():
    # P3: central differences of L = <y, dy> along random directions.
    wl = tiny("basic", 1, n=2, h=4, w=4, c=2)
    st = make_state(wl)
    rng = np.random.default_rng(9)
    x1, x2, dy1, dy2 = rand_io(wl, 5)
    y1, y2 = st.forward(x1, x2)

    def loss(xa, xb, params):
        s2 = StageState(params, st.names, 2)
        a, b = s2.forward(xa, xb)
        return (a * dy1).sum() + (b * dy2).sum()

    # no pre-ReLU value near zero, else the derivative is ill-posed
    _, graph = revblock.function_forward(x2, st._layers(0, 0), st.eps)
    assert np.abs(graph[0][2]).min() > 1e-4
    _, _, dx1, dx2, grads = st.backward(y1, y2, dy1, dy2)
    eps = 1e-6
    for trial in range(3):
        v1, v2 = rng.standard_normal(x1.shape), rng.standard_normal(x2.shape)
        fd = (loss(x1 + eps * v1, x2 + eps * v2, st.params)
              - loss(x1 - eps * v1, x2 - eps * v2, st.params)) / (2 * eps)
        an = (dx1 * v1).sum() + (dx2 * v2).sum()
        assert abs(fd - an) <= 1e-6 * max(abs(an), 1e-8)
        vs = [rng.standard_normal(p.shape) for p in st.params]
        pp = [p + eps * v for p, v in zip(st.params, vs)]
        pm = [p - eps * v for p, v in zip(st.params, vs)]
        fd = (loss(x1, x2, pp) - loss(x1, x2, pm)) / (2 * eps)
        an = sum((g * v).sum() for g, v in zip(grads, vs))
        assert abs(fd - an) <= 1e-6 * max(abs(an), 1e-8)


def test_identity_block_special_case():
    # P5: gamma = beta = 0 on the last BN of F and G makes the block the
    # identity; the only non-zero parameter gradients are those last-BN
    # gamma/beta, equal to sum(dv * xhat) and sum(dv).
    wl = tiny("basic", 1, n=2, h=4, w=4, c=3)
    st = make_state(wl)
    for f in range(2):
        base = f * 6
        st.params[base + 4][:] = 0.0
        st.params[base + 5][:] = 0.0
    x1, x2, dy1, dy2 = rand_io(wl, 8)
    y1, y2 = st.forward(x1, x2)
    assert np.array_equal(y1, x1) and np.array_equal(y2, x2)
    rx1, rx2, dx1, dx2, grads = st.backward(y1, y2, dy1, dy2)
    assert np.array_equal(rx1, y1) and np.array_equal(rx2, y2)
    assert np.array_equal(dx1, dy1) and np.array_equal(dx2, dy2)
    for i, g in enumerate(grads):
        if i % 6 in (4, 5):
            continue
        assert np.abs(g).max() == 0.0
    # last BN of G sees input y1 and upstream dy2; of F: input x2, upstream dy1
    for f, (u, dv) in enumerate(((x2, dy1), (y1, dy2))):
        layers = st._layers(0, f)
        _, graph = revblock.function_forward(u, layers, st.eps)
        xhat = graph[-1][3][0]
        np.testing.assert_allclose(grads[f * 6 + 4], (dv * xhat).sum(axis=(0, 1, 2)), rtol=1e-12)
        np.testing.assert_allclose(grads[f * 6 + 5], dv.sum(axis=(0, 1, 2)), rtol=1e-12)


def test_running_stats_only_in_backward_and_match_torch():
    wl = tiny("basic", 1, n=2, h=4, w=4, c=3)
    st = make_state(wl)
    x1, x2, dy1, dy2 = rand_io(wl, 4)
    y1, y2 = st.forward(x1, x2)
    assert all(np.array_equal(m, 0 * m) for m in st.run_mean)
    assert all(np.array_equal(v, 0 * v + 1) for v in st.run_var)
    st.backward(y1, y2, dy1, dy2)
    # torch: train-mode forward of G on y1 and of F on the reconstructed x2
    for f, u in ((1, y1), (0, x2)):
        base = f * 6
        run = [(torch.zeros(3, dtype=torch.float64), torch.ones(3, dtype=torch.float64)) for _ in range(2)]
        lay = [(oihw(st.params[base + 3 * l]), torch.tensor(st.params[base + 3 * l + 1]),
                torch.tensor(st.params[base + 3 * l + 2])) for l in range(2)]
        residual_fn(nchw(u), lay, running=run)
        for l in range(2):
            slot = (base + 3 * l) // 3
            np.testing.assert_allclose(st.run_mean[slot], run[l][0].numpy(), rtol=1e-10, atol=1e-14)
            np.testing.assert_allclose(st.run_var[slot], run[l][1].numpy(), rtol=1e-10)


def test_storage_hook_points_and_fixed_points():
    # The storage map is applied where tensors are materialised: per function
    # L conv outputs + (L-1) ReLU activations, plus the coupling output.
    wl = tiny("basic", 2, n=2, h=4, w=4, c=4)
    calls = []

    def store(a):
        calls.append(a.shape)
        return synth.round_bf16(a)
    params = [p.astype(np.float64) for p in synth.stage_params(wl, "random")]
    st = StageState(params, [n for n, _ in wl.param_shapes()], 2, store=store)
    x1, x2, dy1, dy2 = (synth.round_bf16(a.astype(np.float32)).astype(np.float64)
                        for a in rand_io(wl, 2))
    y1, y2 = st.forward(x1, x2)
    assert len(calls) == wl.blocks * 2 * (2 + 1 + 1)
    for t in (y1, y2):
        assert np.array_equal(synth.round_bf16(t.astype(np.float32)), t)
    calls.clear()
    rx1, rx2, dx1, dx2, _ = st.backward(y1, y2, dy1, dy2)
    # per function: recompute (2 h + 1 act) + reconstruction + output gradient
    # + dh of both layers + dz of the inner layer
    assert len(calls) == wl.blocks * 2 * (3 + 1 + 1 + 2 + 1)
    for t in (rx1, rx2, dx1, dx2):
        assert np.array_equal(synth.round_bf16(t.astype(np.float32)), t)
    # the bf16-stored result stays near the fp64 one
    ref = make_state(wl)
    ry1, ry2 = ref.forward(x1, x2)
    assert np.linalg.norm(y1 - ry1) <= 1e-2 * np.linalg.norm(ry1)
    assert np.linalg.norm(rx1 - x1) <= 5e-2 * np.linalg.norm(x1)


@pytest.mark.parametrize("kind", ["basic", "bottleneck"])
def test_block_vjp_from_stored_input_equals_backprop(kind):
    # The input-buffer variant's block VJP (no reconstruction) against torch
    # autograd through the block at the same input and parameters.
    wl = tiny(kind, 1, n=2, h=5, w=4, c=4, mid=3)
    st = make_state(wl)
    x1, x2, dy1, dy2 = rand_io(wl, 5)
    ty1, ty2, tdx1, tdx2, tgrads = torch_stage_grads(wl, st, x1, x2, dy1, dy2)
    r = revblock.block_vjp(x1, x2, dy1, dy2, st._layers(0, 0), st._layers(0, 1), st.eps)
    np.testing.assert_allclose(r["dx1"], tdx1, rtol=1e-10, atol=1e-12)
    np.testing.assert_allclose(r["dx2"], tdx2, rtol=1e-10, atol=1e-12)
    got = [t for f in ("dF", "dG") for trip in r[f] for t in trip]
    for g, tg in zip(got, tgrads):
        assert np.linalg.norm(g - tg) <= 1e-10 * max(np.linalg.norm(tg), 1e-30)
