"""Independent PyTorch-CPU (fp64) formulation of the block, used only to pin
the oracle: a library special case written directly from the definitions
(torch conv2d / batch_norm / relu with autograd), sharing no code with it."""
import torch
import torch.nn.functional as Fn


def nchw(x):
    return torch.as_tensor(x, dtype=torch.float64).permute(0, 3, 1, 2)


def nhwc(t):
    return t.permute(0, 2, 3, 1)


def oihw(w):
    return torch.as_tensor(w, dtype=torch.float64).permute(0, 3, 1, 2)


def residual_fn(u, layers, eps=1e-5, running=None):
    """u: NCHW tensor; layers: list of (W OIHW, gamma, beta) tensors."""
    a = u
    for l, (w, g, b) in enumerate(layers):
        pad = (w.shape[-1] - 1) // 2
        h = Fn.conv2d(a, w, padding=pad)
        rm = rv = None
        if running is not None:
            rm, rv = running[l]
        o = Fn.batch_norm(h, rm, rv, g, b, training=True, momentum=0.1, eps=eps)
        a = o if l == len(layers) - 1 else torch.relu(o)
    return a


def block(x1, x2, fl, gl, eps=1e-5):
    y1 = x1 + residual_fn(x2, fl, eps)
    y2 = x2 + residual_fn(y1, gl, eps)
    return y1, y2


def front(x, P, j):
    """Non-reversible layer that opens stage j (NCHW): the stem on the images or
    the stride-2 downsampling."""
    if j == 0:
        w = P["s0.stem.weight"].permute(0, 3, 1, 2)
        h = Fn.conv2d(x, w, padding=1)
        return torch.relu(Fn.batch_norm(h, None, None, P["s0.stem_bn.gamma"],
                                        P["s0.stem_bn.beta"], training=True, eps=1e-5))
    w = P[f"s{j}.trans.weight"].permute(0, 3, 1, 2)
    h = Fn.conv2d(x, w, stride=2)
    return Fn.batch_norm(h, None, None, P[f"s{j}.trans_bn.gamma"], P[f"s{j}.trans_bn.beta"],
                         training=True, eps=1e-5)


def stage_blocks(x1, x2, P, j, blocks):
    for b in range(blocks):
        def lay(f):
            return [(P[f"s{j}.b{b}.{f}.conv{l}.weight"].permute(0, 3, 1, 2),
                     P[f"s{j}.b{b}.{f}.bn{l}.gamma"], P[f"s{j}.b{b}.{f}.bn{l}.beta"]) for l in range(2)]
        x1, x2 = block(x1, x2, lay("F"), lay("G"))
    return x1, x2


def revnet(img_nhwc, params, names, stages, blocks):
    """Whole network in torch (NCHW inside), params as torch leaves in canonical order."""
    P = dict(zip(names, params))
    x = nchw(img_nhwc) if not isinstance(img_nhwc, torch.Tensor) else img_nhwc
    for j in range(stages):
        x = front(x, P, j)
        c = x.shape[1] // 2
        x1, x2 = stage_blocks(x[:, :c], x[:, c:], P, j, blocks)
        x = torch.cat([x1, x2], dim=1)
    pooled = x.mean(dim=(2, 3))
    J = stages - 1
    return pooled @ P[f"s{J}.fc.weight"].T + P[f"s{J}.fc.bias"]
