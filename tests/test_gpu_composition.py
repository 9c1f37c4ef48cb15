"""A stage of B blocks is the composition of its blocks (Sec. 3.2: the stage
map is the blocks applied in sequence; its inverse runs them in reverse).  At
the workloads' full sizes, in the launch configuration the benchmark times
(petra_stage_step), the B-block stage must give bit for bit what B one-block
stages give when chained by hand: the forward output, the reconstructed input
and the running statistics (which the recompute of each block produces).

The gradient side is not compared bit for bit: across a block boundary the
stage's backward forms the next function's BN-backward partial sums in the
epilogue of the kernel that writes the input gradient, while a one-block
stage forms them from its input gradient in a pass of its own, so the same
sums are added in another order (it is covered against the oracle by the
parity tests)."""
import numpy as np
import pytest

import synth
from tests.harness import gpu_stage

pytestmark = pytest.mark.gpu


def _block_params(wl, params, b):
    per = len(params) // wl.blocks
    return params[b * per:(b + 1) * per]


@pytest.mark.parametrize("wl", [synth.CIFAR_STAGE, synth.IMAGENET32_STAGE,
                                synth.IMAGENET_BOTTLENECK_STAGE,
                                synth.CIFAR_STAGE.with_(dtype="fp32", n=16)],
                         ids=["cifar_stage", "imagenet32_stage", "imagenet_bottleneck_stage",
                              "cifar_fp32_16"])
def test_stage_is_composition_of_blocks_bitwise(wl):
    import torch
    from paper_2406_02052_amd import to_host

    print(f"composition case {wl.name} {wl.dtype} n={wl.n}", flush=True)
    params = synth.stage_params(wl, "random")
    xa = synth.stage_input(wl)
    yb = synth.stage_input(wl, seed_offset=10)
    g = synth.stage_output_grad(wl)

    # the whole stage through one petra_stage_step (forward || backward, update)
    st = gpu_stage(wl, params)
    xa1, xa2 = st.act(xa[0]), st.act(xa[1])
    yb1, yb2, g1, g2 = st.act(yb[0]), st.act(yb[1]), st.act(g[0]), st.act(g[1])
    ya1, ya2, xr1, xr2, dx1, dx2 = (st.act() for _ in range(6))
    assert st.step(xa1, xa2, ya1, ya2, yb1, yb2, g1, g2, xr1, xr2, dx1, dx2)
    torch.cuda.synchronize()
    whole = {"y1": to_host(ya1), "y2": to_host(ya2), "x1": to_host(xr1), "x2": to_host(xr2),
             "dx1": to_host(dx1), "dx2": to_host(dx2)}
    n_bn = st.n_bn // wl.blocks
    rmean, rvar = st.run_mean.cpu().numpy(), st.run_var.cpu().numpy()
    del st

    # the same step block by block: forward 0..B-1, backward B-1..0
    blocks = [gpu_stage(wl.with_(blocks=1), _block_params(wl, params, b)) for b in range(wl.blocks)]
    s0 = blocks[0]
    u1, u2 = s0.act(xa[0]), s0.act(xa[1])
    for blk in blocks:
        v1, v2 = blk.act(), blk.act()
        blk.forward(u1, u2, v1, v2)
        u1, u2 = v1, v2
    r1, r2, d1, d2 = s0.act(yb[0]), s0.act(yb[1]), s0.act(g[0]), s0.act(g[1])
    for blk in reversed(blocks):
        o1, o2, e1, e2 = (blk.act() for _ in range(4))
        blk.reconstruct_backward(r1, r2, d1, d2, o1, o2, e1, e2)
        r1, r2, d1, d2 = o1, o2, e1, e2
    torch.cuda.synchronize()
    chained = {"y1": to_host(u1), "y2": to_host(u2), "x1": to_host(r1), "x2": to_host(r2),
               "dx1": to_host(d1), "dx2": to_host(d2)}
    for k in ("y1", "y2", "x1", "x2"):
        assert np.array_equal(whole[k], chained[k]), f"{k} differs from the chained blocks"
    for b, blk in enumerate(blocks):
        bsl = slice(b * n_bn, (b + 1) * n_bn)
        assert np.array_equal(rmean[bsl], blk.run_mean.cpu().numpy()), f"block {b} running mean"
        assert np.array_equal(rvar[bsl], blk.run_var.cpu().numpy()), f"block {b} running var"
