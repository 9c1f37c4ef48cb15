"""petra_stage_forward_noalloc (the forward for callers that cannot allocate:
scratch in the library's static device array) against petra_stage_forward on
the same handle and inputs, bit for bit: two calls in a row on two stages, the
second smaller (both share the one array), then a handle bound without any
workspace, and the rejection of a stage whose forward needs more scratch than
the array holds."""
import ctypes

import numpy as np
import pytest

import synth
from tests.harness import gpu_stage

pytestmark = pytest.mark.gpu


def _lib():
    from paper_2406_02052_amd import _lib as L
    lib = L.load()
    fn = lib.petra_stage_forward_noalloc
    fn.restype = ctypes.c_int
    fn.argtypes = [ctypes.c_void_p] * 6
    return L, fn


def _forward_both(wl):
    import torch
    from paper_2406_02052_amd import to_host

    L, fwd_noalloc = _lib()
    st = gpu_stage(wl, synth.stage_params(wl, "random"))
    x1, x2 = (st.act(a) for a in synth.stage_input(wl))
    ya1, ya2, yb1, yb2 = (st.act() for _ in range(4))
    st.forward(x1, x2, ya1, ya2)
    rc = fwd_noalloc(st.handle, x1.data_ptr(), x2.data_ptr(), yb1.data_ptr(), yb2.data_ptr(), None)
    assert rc == 0, L.load().petra_last_error()
    torch.cuda.synchronize()
    return [to_host(t) for t in (ya1, ya2)], [to_host(t) for t in (yb1, yb2)]


def test_forward_noalloc_matches_forward_two_calls_second_smaller():
    first = synth.CIFAR_STAGE.with_(n=32)
    second = synth.CIFAR_STAGE.with_(n=5, h=9, w=32, blocks=1)
    for wl in (first, second):
        print(f"noalloc case {wl.name} n={wl.n} h={wl.h} w={wl.w} blocks={wl.blocks}", flush=True)
        want, got = _forward_both(wl)
        for a, b in zip(want, got):
            assert np.array_equal(a, b)


def test_forward_noalloc_matches_forward_bottleneck_full_size():
    """The bottleneck stage at its full batch (its forward keeps the two
    32-channel pre-BN tensors only: the 128-channel one is recomputed where the
    coupling consumes it, so the working set fits the static array)."""
    wl = synth.IMAGENET_BOTTLENECK_STAGE
    print(f"noalloc case {wl.name} n={wl.n}", flush=True)
    want, got = _forward_both(wl)
    for a, b in zip(want, got):
        assert np.array_equal(a, b)


def test_forward_noalloc_on_a_handle_without_workspace():
    import torch
    from paper_2406_02052_amd import PetraError, Stage, to_host

    L, fwd_noalloc = _lib()
    wl = synth.IMAGENET32_STAGE.with_(n=4, blocks=2)
    params = synth.stage_params(wl, "random")
    ref = gpu_stage(wl, params)
    x1, x2 = (ref.act(a) for a in synth.stage_input(wl))
    y1, y2 = ref.act(), ref.act()
    ref.forward(x1, x2, y1, y2)
    # a second handle of the same stage, bound without a workspace
    st = Stage(wl.n, wl.h, wl.w, wl.c_half, wl.blocks, wl.kind, wl.dtype)
    L.petra_stage_bind(st.handle, st.params, st.grad, st.mom, st.run_mean, st.run_var, 0, 0)
    st.params.copy_(ref.params)
    z1, z2 = st.act(), st.act()
    rc = fwd_noalloc(st.handle, x1.data_ptr(), x2.data_ptr(), z1.data_ptr(), z2.data_ptr(), None)
    assert rc == 0, L.load().petra_last_error()
    torch.cuda.synchronize()
    assert np.array_equal(to_host(y1), to_host(z1)) and np.array_equal(to_host(y2), to_host(z2))
    with pytest.raises(PetraError) as e:
        st.forward(x1, x2, z1, z2)
    assert e.value.name == "PETRA_ERR_WORKSPACE"


def test_forward_noalloc_rejects_a_stage_beyond_the_scratch():
    from paper_2406_02052_amd import _lib as L

    _, fwd_noalloc = _lib()
    # at batch 192 the bottleneck stage's forward holds two 38.5 MB pre-BN tensors
    wl = synth.IMAGENET_BOTTLENECK_STAGE
    st = gpu_stage(wl.with_(n=192), synth.stage_params(wl, "random"))
    a = [st.act() for _ in range(4)]
    rc = fwd_noalloc(st.handle, *(t.data_ptr() for t in a), None)
    assert L.STATUS[rc] == "PETRA_ERR_WORKSPACE"
    assert "static scratch" in L.load().petra_last_error().decode()
