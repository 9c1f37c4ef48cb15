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
