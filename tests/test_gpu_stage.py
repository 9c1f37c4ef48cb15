"""GPU parity of the reversible stage step against the oracle (through the C ABI)."""
import numpy as np
import pytest

import synth
from tests.harness import check, gpu_stage, run_step_parity

pytestmark = pytest.mark.gpu

SMALL = {
    # exact workload of the fp32 single-block case
    "fp32_block_8x8x8x32": synth.BLOCK_FP32,
    # one partial tile, ragged reduction (K = 144), two blocks
    "fp32_ragged_3x7x5_c16": synth.BLOCK_FP32.with_(n=3, h=7, w=5, blocks=2),
    "fp32_3tiles_5x9x7_c32": synth.BLOCK_FP32.with_(n=5, h=9, w=7, c_half=32, blocks=1),
    "fp32_bottleneck_2x6x6": synth.BLOCK_FP32.with_(n=2, h=6, w=6, c_half=32, c_mid=16,
                                                     kind="bottleneck", blocks=1),
    # BN over two rows: the variance must not come from E[h^2] - E[h]^2
    "fp32_two_rows_2x1x1": synth.BLOCK_FP32.with_(n=2, h=1, w=1, blocks=2),
    "fp32_three_rows_3x1x1_c64": synth.BLOCK_FP32.with_(n=3, h=1, w=1, c_half=64, blocks=1),
    # fp32 twins of the bf16 stage shapes (same kernels' structure, 1e-4)
    "fp32_c32_4x9x9": synth.CIFAR_STAGE.with_(n=4, h=9, w=9, dtype="fp32"),
    "fp32_c128_3x6x6": synth.IMAGENET32_STAGE.with_(n=3, h=6, w=6, blocks=2, dtype="fp32"),
    "fp32_bottleneck_2x12x12": synth.IMAGENET_BOTTLENECK_STAGE.with_(n=2, h=12, w=12, blocks=2,
                                                                      dtype="fp32"),
    "bf16_c32_4x9x9": synth.CIFAR_STAGE.with_(n=4, h=9, w=9),
    "bf16_c64_2x10x10": synth.CIFAR_STAGE.with_(n=2, h=10, w=10, c_half=64, blocks=1),
    "bf16_c128_3x6x6": synth.IMAGENET32_STAGE.with_(n=3, h=6, w=6, blocks=2),
    "bf16_bottleneck_2x12x12": synth.IMAGENET_BOTTLENECK_STAGE.with_(n=2, h=12, w=12, blocks=2),
    "bf16_c256_2x4x4": synth.IMAGENET32_STAGE.with_(n=2, h=4, w=4, c_half=256, blocks=1),
    # halo-tile conv shapes (image widths 32 / 16 / 56), with ragged row tiles
    "bf16_halo_c32_2x5x32": synth.CIFAR_STAGE.with_(n=2, h=5, w=32),
    "bf16_halo_c64_2x9x16": synth.CIFAR_STAGE.with_(n=2, h=9, w=16, c_half=64, blocks=1),
    "bf16_halo_c128_1x9x16": synth.IMAGENET32_STAGE.with_(n=1, h=9, w=16, blocks=2),
    "bf16_halo_bottleneck_1x5x56": synth.IMAGENET_BOTTLENECK_STAGE.with_(n=1, h=5, w=56, blocks=1),
    # whole-image conv (16x16, 128 channels: one workgroup per image) and the
    # weight gradient that splits the 9 taps over three waves, at batches of
    # one and two images (the weight gradient then has as many splits as tiles)
    "bf16_img_c128_2x16x16": synth.IMAGENET32_STAGE.with_(n=2, h=16, w=16, blocks=2),
    "bf16_img_c128_1x16x16": synth.IMAGENET32_STAGE.with_(n=1, h=16, w=16, blocks=1),
    # streaming 1x1 convs (128 -> 32, 32 -> 128): 1587 pixels = 100 units of 16
    # (the last one 3 pixels) over 25 workgroups; 18769 pixels = 1174 units (the
    # last one a single pixel) over the full 256-workgroup grid, 1-2 units a wave
    "bf16_bottleneck_1x1_3x23x23": synth.IMAGENET_BOTTLENECK_STAGE.with_(n=3, h=23, w=23,
                                                                          blocks=1),
    "bf16_bottleneck_1x1_1x137x137": synth.IMAGENET_BOTTLENECK_STAGE.with_(n=1, h=137, w=137,
                                                                            blocks=1),
}


def _small_cases():
    """Every small case in full coupling; the bf16 ones also with one function
    isolated (the other's last BN zeroed), which differentiates one function
    at a time and so holds the stated bar."""
    out = []
    for name, wl in SMALL.items():
        out.append((name, "full"))
        if wl.dtype == "bf16":
            out += [(name, "isoF"), (name, "isoG")]
    return out


@pytest.mark.parametrize("name,mode", _small_cases())
def test_stage_step_parity_small(name, mode):
    wl = SMALL[name]
    print(f"case {name} {mode}: {wl}", flush=True)
    got, want, exact = run_step_parity(wl, bn_affine="random", mode=mode)
    print(check(wl, mode, got, want, exact), flush=True)


@pytest.mark.parametrize("name", ["fp32_block_8x8x8x32", "bf16_c32_4x9x9", "bf16_c128_3x6x6",
                                  "bf16_bottleneck_2x12x12"])
def test_identity_block_small(name):
    """P5 (Eq. 4): with gamma = beta = 0 on the last BN of F and of G every block
    is the identity; the step must return its inputs bit for bit and only the
    last BNs' parameters get a gradient (their sums of dy and dy * xhat)."""
    wl = SMALL[name]
    got, want, exact = run_step_parity(wl, bn_affine="random", mode="p5")
    print(check(wl, "p5", got, want, exact), flush=True)


def test_fp32_block_unit_bn_affine():
    """The exact single-block fp32 workload with BN gamma = 1, beta = 0."""
    wl = synth.BLOCK_FP32
    got, want, exact = run_step_parity(wl, bn_affine="identity")
    print(check(wl, "full", got, want, exact), flush=True)


def _io(st, wl, seed):
    rng = np.random.default_rng(seed)
    shp = (wl.n, wl.h, wl.w, wl.c_half)
    return [st.act(synth.to_storage(rng.standard_normal(shp, dtype=np.float32), wl.dtype))
            for _ in range(4)]


def test_step_concurrent_equals_sequential_bitwise():
    """petra_stage_step (forward and backward on two streams) must give the same
    bits as the forward, backward and update issued one after another, and
    repeated runs must be bitwise identical (deterministic reductions)."""
    import torch
    from paper_2406_02052_amd import to_host

    wl = synth.CIFAR_STAGE.with_(n=8, h=16, w=16)
    params = synth.stage_params(wl, "random")
    outs = []
    for mode in ("seq", "step", "step"):
        st = gpu_stage(wl, params)
        xa1, xa2, _, _ = _io(st, wl, 1)
        yb1, yb2, db1, db2 = _io(st, wl, 2)
        ya1, ya2, xb1, xb2, dxb1, dxb2 = (st.act() for _ in range(6))
        for _ in range(2):
            if mode == "seq":
                st.forward(xa1, xa2, ya1, ya2)
                st.reconstruct_backward(yb1, yb2, db1, db2, xb1, xb2, dxb1, dxb2)
                st.update()
            else:
                st.step(xa1, xa2, ya1, ya2, yb1, yb2, db1, db2, xb1, xb2, dxb1, dxb2)
        torch.cuda.synchronize()
        outs.append([to_host(t) for t in (ya1, ya2, xb1, xb2, dxb1, dxb2)] +
                    [st.params.cpu().numpy(), st.mom.cpu().numpy(), st.run_mean.cpu().numpy(),
                     st.run_var.cpu().numpy()])
    for a, b, c in zip(*outs):
        assert np.array_equal(a, b) and np.array_equal(b, c)


def test_in_place_aliasing_matches_out_of_place():
    import torch
    from paper_2406_02052_amd import to_host

    wl = synth.IMAGENET32_STAGE.with_(n=2, h=8, w=8, c_half=64, blocks=2)
    params = synth.stage_params(wl, "random")
    res = []
    for inplace in (False, True):
        st = gpu_stage(wl, params)
        a1, a2, g1, g2 = _io(st, wl, 5)
        if inplace:
            st.forward(a1, a2, a1, a2)
            st.reconstruct_backward(a1, a2, g1, g2, a1, a2, g1, g2)
            outs = (a1, a2, g1, g2)
        else:
            y1, y2, x1, x2, d1, d2 = (st.act() for _ in range(6))
            st.forward(a1, a2, y1, y2)
            st.reconstruct_backward(y1, y2, g1, g2, x1, x2, d1, d2)
            outs = (x1, x2, d1, d2)
        torch.cuda.synchronize()
        res.append([to_host(t) for t in outs] + [st.grad.cpu().numpy()])
    for a, b in zip(*res):
        assert np.array_equal(a, b)


def test_accumulation_k_updates_every_kth_backward():
    import torch

    wl = synth.CIFAR_STAGE.with_(n=2, h=8, w=8, accum_k=3)
    params = synth.stage_params(wl, "random")
    st = gpu_stage(wl, params)
    y1, y2, g1, g2 = _io(st, wl, 7)
    x1, x2, d1, d2 = (st.act() for _ in range(4))
    fired = []
    for _ in range(6):
        st.reconstruct_backward(y1, y2, g1, g2, x1, x2, d1, d2)
        fired.append(st.update())
    torch.cuda.synchronize()
    assert fired == [False, False, True, False, False, True]


def test_graph_replay_matches_eager_every_replay():
    """The cached-graph path must give the eager path's bits on every replay,
    with unrelated eager work and synchronisations between the replays."""
    import torch
    from paper_2406_02052_amd import to_host

    wl = synth.CIFAR_STAGE.with_(n=4, h=8, w=32)
    params = synth.stage_params(wl, "random")
    stages = []
    for graphs in (False, True):
        st = gpu_stage(wl, params)
        st.set_graphs(graphs)
        stages.append((st, _io(st, wl, 11), _io(st, wl, 12)))
    scratch = torch.zeros(1 << 20, device="cuda")
    for rep in range(3):
        outs = []
        for st, (xa1, xa2, _, _), (yb1, yb2, db1, db2) in stages:
            ya1, ya2, xb1, xb2, dxb1, dxb2 = (st.act() for _ in range(6))
            if rep == 2:
                st.forward(xa1, xa2, ya1, ya2)
                st.reconstruct_backward(yb1, yb2, db1, db2, xb1, xb2, dxb1, dxb2)
                st.update()
            else:
                st.step(xa1, xa2, ya1, ya2, yb1, yb2, db1, db2, xb1, xb2, dxb1, dxb2)
            scratch.add_(1.0)           # unrelated eager work between replays
            torch.cuda.synchronize()
            outs.append([to_host(t) for t in (ya1, ya2, xb1, xb2, dxb1, dxb2)] +
                        [st.params.cpu().numpy(), st.mom.cpu().numpy(), st.run_var.cpu().numpy()])
        for a, b in zip(*outs):
            assert np.array_equal(a, b), f"replay {rep} differs from eager"


@pytest.mark.parametrize("wl_name,shape", [
    ("cifar", dict(n=4, h=8, w=32)),
    ("bottleneck", dict(n=1, h=5, w=56, blocks=2)),
])
def test_backward_stream_modes_bitwise(wl_name, shape):
    """One, two or three streams per backward (and graph replay of the
    three-stream program) must give identical bits: the cross-stream ordering
    covers every read-after-write and in-place hazard."""
    import torch
    from paper_2406_02052_amd import to_host

    base = synth.CIFAR_STAGE if wl_name == "cifar" else synth.IMAGENET_BOTTLENECK_STAGE
    wl = base.with_(**shape)
    params = synth.stage_params(wl, "random")
    res = []
    for streams, graphs in ((1, False), (2, False), (3, False), (3, True)):
        st = gpu_stage(wl, params)
        st.set_streams(streams)
        st.set_graphs(graphs)
        a1, a2, g1, g2 = _io(st, wl, 21)
        for _ in range(2):   # in place: y -> x and dy -> dx in the same buffers
            st.reconstruct_backward(a1, a2, g1, g2, a1, a2, g1, g2)
            st.update()
        torch.cuda.synchronize()
        res.append([to_host(t) for t in (a1, a2, g1, g2)] +
                   [st.params.cpu().numpy(), st.run_mean.cpu().numpy(), st.run_var.cpu().numpy()])
    for mode in res[1:]:
        for a, b in zip(res[0], mode):
            assert np.array_equal(a, b)
