"""Pins of the oracle's bf16 storage model.

Reading (bf16 workloads: bf16 storage, fp32 accumulation).  Every tensor a
bf16 implementation of the reversible step materialises is held at bf16: the
pre-BN conv outputs (whose batch statistics BN takes), the ReLU activations a
conv consumes, the coupling outputs (y, the reconstructed x, the input
gradients) and the gradients dz (after a ReLU mask) and dh (out of a BN
backward); the arithmetic in between is exact (fp64 here).  The ReLU
decisions are thereby taken on stored values.

The oracle applies that rule through its `store` hook.  This file pins it
against a formulation that shares nothing with the oracle: torch-CPU conv2d /
batch_norm / relu in fp64, torch's own bf16 conversion at the points named
above (as autograd functions that round the value in the forward or the
gradient in the backward), and torch autograd for the vector-Jacobian
products, with the reconstruction of Eq. 4 written out.  Stored tensors must
agree bit for bit and the parameter gradients to fp64 rounding; a rounding
placed at another point, or a missing one, moves many stored values by an
ulp and fails."""
import numpy as np
import pytest
import torch
import torch.nn.functional as Fn

import synth
from oracle.stage import StageState
from tests.torch_ref import nchw, nhwc


def bf(t):
    """fp64 -> fp32 -> bf16 -> fp64 with torch's conversions (nearest even)."""
    return t.to(torch.float32).to(torch.bfloat16).to(torch.float64)


class StoreValue(torch.autograd.Function):
    """Forward: the value as stored in bf16; backward: the gradient unchanged."""
    @staticmethod
    def forward(ctx, x):
        return bf(x)

    @staticmethod
    def backward(ctx, g):
        return g


class StoreGrad(torch.autograd.Function):
    """Forward: unchanged; backward: the gradient as stored in bf16."""
    @staticmethod
    def forward(ctx, x):
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return bf(g)


def fn_bf16(u, layers, eps):
    """Residual function with bf16 storage: conv -> store(h) (its gradient dh
    stored too) -> BN -> [ReLU, dz stored, activation stored] ... -> BN."""
    a = u
    for l, (w, g, b) in enumerate(layers):
        h = Fn.conv2d(a, w, padding=(w.shape[-1] - 1) // 2)
        h = StoreGrad.apply(StoreValue.apply(h))
        o = Fn.batch_norm(h, None, None, g, b, training=True, eps=eps)
        if l == len(layers) - 1:
            a = o
        else:
            a = StoreValue.apply(torch.relu(StoreGrad.apply(o)))
    return a


def torch_block_step(y1, y2, g1, g2, f_layers, g_layers, eps):
    """Reconstruct + VJP of one block (Eq. 4, Eq. 5) with bf16 storage.
    Inputs NCHW fp64 (bf16-representable); layers: [(W OIHW, gamma, beta)] as
    leaves requiring grad.  Returns x1, x2, dx1, dx2 and the parameter
    gradients of F then G in canonical order."""
    y1l = y1.clone().requires_grad_(True)
    gout = fn_bf16(y1l, g_layers, eps)
    x2 = bf(y2 - gout.detach())
    gp = [t for lay in g_layers for t in lay]
    grads_g = torch.autograd.grad(gout, [y1l] + gp, grad_outputs=g2)
    z1 = bf(g1 + grads_g[0])
    x2l = x2.clone().requires_grad_(True)
    fout = fn_bf16(x2l, f_layers, eps)
    x1 = bf(y1 - fout.detach())
    fp = [t for lay in f_layers for t in lay]
    grads_f = torch.autograd.grad(fout, [x2l] + fp, grad_outputs=z1)
    dx2 = bf(g2 + grads_f[0])
    return x1, x2, z1, dx2, list(grads_f[1:]) + list(grads_g[1:])


def torch_block_forward(x1, x2, f_layers, g_layers, eps):
    with torch.no_grad():
        y1 = bf(x1 + fn_bf16(x2, f_layers, eps))
        y2 = bf(x2 + fn_bf16(y1, g_layers, eps))
    return y1, y2


def layers_of(params, base, n_convs, weight_bf16):
    out = []
    for l in range(n_convs):
        w, g, b = params[base + 3 * l: base + 3 * l + 3]
        w = torch.as_tensor(w, dtype=torch.float64)
        if weight_bf16:
            w = bf(w)
        out.append((w.permute(0, 3, 1, 2).contiguous().requires_grad_(True),
                    torch.as_tensor(g, dtype=torch.float64).clone().requires_grad_(True),
                    torch.as_tensor(b, dtype=torch.float64).clone().requires_grad_(True)))
    return out


CASES = {
    "basic_2blocks": synth.StageWorkload("pin", "bf16", 2, 6, 5, 8, "basic", 2,
                                         x_dist="normal", dy_sigma=1.0),
    "bottleneck_1block": synth.StageWorkload("pin", "bf16", 2, 5, 6, 8, "bottleneck", 1, c_mid=4,
                                             x_dist="abs_normal", dy_sigma=1e-2),
}


@pytest.mark.parametrize("name", list(CASES))
def test_storage_oracle_equals_torch_bf16_formulation(name):
    wl = CASES[name]
    params = synth.stage_params(wl, "random")
    names = [n for n, _ in wl.param_shapes()]
    nconv = len(wl.conv_layers())
    x1, x2 = synth.stage_input(wl)
    g1, g2 = synth.stage_output_grad(wl)
    ref = StageState(params, names, nconv, weight_view=synth.round_bf16, store=synth.round_bf16)
    oy1, oy2 = ref.forward(x1, x2)
    ox1, ox2, odx1, odx2, ograds = ref.backward(oy1, oy2, g1, g2)

    per_fn = 3 * nconv
    lay = [[layers_of(params, (2 * b + f) * per_fn, nconv, True) for f in (0, 1)]
           for b in range(wl.blocks)]
    t1, t2 = nchw(x1), nchw(x2)
    for b in range(wl.blocks):
        t1, t2 = torch_block_forward(t1, t2, lay[b][0], lay[b][1], 1e-5)
    for a, b in ((nhwc(t1).numpy(), oy1), (nhwc(t2).numpy(), oy2)):
        assert np.array_equal(a, b), "forward output differs from the storage oracle"
    r1, r2, d1, d2 = t1, t2, nchw(g1), nchw(g2)
    tgrads = [None] * len(params)
    for b in reversed(range(wl.blocks)):
        r1, r2, d1, d2, gr = torch_block_step(r1, r2, d1, d2, lay[b][0], lay[b][1], 1e-5)
        for i, gtensor in enumerate(gr):
            f, rest = divmod(i, per_fn)
            idx = (2 * b + f) * per_fn + rest
            if rest % 3 == 0:
                gtensor = gtensor.permute(0, 2, 3, 1)  # OIHW -> KRSC
            tgrads[idx] = gtensor.detach().numpy()
    for a, b, nm in ((nhwc(r1).detach().numpy(), ox1, "x1"), (nhwc(r2).detach().numpy(), ox2, "x2"),
                     (nhwc(d1).detach().numpy(), odx1, "dx1"), (nhwc(d2).detach().numpy(), odx2, "dx2")):
        assert np.array_equal(a, b), f"{nm} differs from the storage oracle"
    for nm, a, b in zip(names, tgrads, ograds):
        scale = max(float(np.abs(b).max()), 1e-30)
        assert float(np.abs(a - b).max()) <= 1e-9 * scale, nm


def test_storage_model_moves_results_by_storage_noise_only():
    """The storage model stays within bf16 storage noise of plain fp64 on a
    single half-coupling (G's last BN zeroed, so the block is y1 = x1 + F(x2)
    and nothing is reconstructed through a long chain): forward output and
    reconstruction at a few bf16 ulps, gradients within 2e-2."""
    wl = CASES["basic_2blocks"].with_(n=4, h=8, w=8, blocks=1)
    params = synth.stage_params(wl, "random")
    names = [n for n, _ in wl.param_shapes()]
    for i, nm in enumerate(names):
        if nm.startswith("b0.G.bn1."):
            params[i] = np.zeros_like(params[i])
    x1, x2 = synth.stage_input(wl)
    g1, g2 = synth.stage_output_grad(wl)
    runs = []
    for store in (synth.round_bf16, None):
        st = StageState(params, names, 2, weight_view=synth.round_bf16, store=store)
        y = st.forward(x1, x2)
        yin = tuple(synth.round_bf16(np.asarray(t, np.float32)) for t in y)
        runs.append((y, st.backward(*yin, g1, g2)))
    (ys, bs), (yp, bp) = runs
    rel = lambda a, b: float(np.linalg.norm(np.asarray(a) - b) / np.linalg.norm(b))
    assert rel(ys[0], yp[0]) < 2 ** -7
    assert np.array_equal(ys[1], x2)          # G = 0: y2 = x2 exactly
    assert np.array_equal(bs[1], ys[1])       # and its reconstruction x2 = y2 - 0
    assert rel(bs[0], bp[0]) < 2 ** -7
    for a, b in zip(bs[4], bp[4]):
        if np.linalg.norm(b) > 0:
            assert rel(a, b) < 2e-2
