"""Host-side checks of the C ABI (no GPU work is launched): the library loads,
exports every symbol its header declares, and validates arguments."""
import ctypes
import glob
import os
import re

import pytest

import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def declared_symbols():
    names = set()
    for h in glob.glob(os.path.join(ROOT, "include", "*.h")):
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"\b(petra_\w+)\s*\(", text))
    return sorted(names)


def test_library_exports_every_declared_symbol():
    from paper_2406_02052_amd import _lib
    lib = ctypes.CDLL(_lib.LIB_PATH)
    syms = declared_symbols()
    assert len(syms) >= 12
    missing = [s for s in syms if not hasattr(lib, s)]
    assert not missing, missing


def _desc(wl):
    from paper_2406_02052_amd import _lib as L
    return L.StageDesc(wl.n, wl.h, wl.w, wl.c_half, wl.c_mid, wl.blocks,
                       0 if wl.kind == "basic" else 1, 1 if wl.dtype == "bf16" else 0,
                       wl.bn_eps, wl.bn_momentum)


@pytest.mark.parametrize("wl,n_params", [(synth.BLOCK_FP32, 9344), (synth.CIFAR_STAGE, 74240),
                                         (synth.IMAGENET32_STAGE, 3545088),
                                         (synth.IMAGENET_BOTTLENECK_STAGE, 106752)])
def test_param_layout(wl, n_params):
    from paper_2406_02052_amd import _lib as L
    h = L.petra_stage_create(_desc(wl))
    try:
        np_, nt, nbn, ws = L.petra_stage_query(h)
        assert np_ == n_params
        shapes = wl.param_shapes()
        assert nt == len(shapes)
        spans = []
        for i, (name, shp) in enumerate(shapes):
            info = L.petra_stage_param_info(h, i)
            assert tuple(info.shape[:info.ndim]) == shp, name
            assert info.weight_decay == (1 if name.endswith("weight") else 0)
            spans.append((info.offset, info.offset + info.numel))
        spans.sort()
        assert spans[0][0] == 0 and spans[-1][1] == n_params
        assert all(a[1] == b[0] for a, b in zip(spans, spans[1:]))
        # all decayed (conv) weights precede the BN parameters
        last_w = max(L.petra_stage_param_info(h, i).offset for i in range(nt) if i % 3 == 0)
        first_bn = min(L.petra_stage_param_info(h, i).offset for i in range(nt) if i % 3 != 0)
        assert last_w < first_bn
        assert nbn == sum(s[0] for n, s in shapes if n.endswith("gamma"))
        assert ws > 0
        with pytest.raises(L.PetraError):
            L.petra_stage_param_info(h, nt)
    finally:
        L.petra_stage_destroy(h)


@pytest.mark.parametrize("field,value,status", [
    ("dtype", 7, "PETRA_ERR_DTYPE"), ("kind", 5, "PETRA_ERR_INVALID_ARG"),
    ("c_half", 24, "PETRA_ERR_SHAPE"), ("c_half", 1024, "PETRA_ERR_SHAPE"),
    ("n", 0, "PETRA_ERR_SHAPE"), ("num_blocks", 0, "PETRA_ERR_SHAPE"),
    ("bn_eps", 0.0, "PETRA_ERR_INVALID_ARG")])
def test_create_rejects_bad_descriptions(field, value, status):
    from paper_2406_02052_amd import _lib as L
    d = _desc(synth.CIFAR_STAGE)
    setattr(d, field, value)
    with pytest.raises(L.PetraError) as e:
        L.petra_stage_create(d)
    assert e.value.name == status
    assert L.petra_last_error() != ""


def test_create_enforces_the_32_bit_buffer_offset_limit():
    """Every kernel addresses activations through buffer resources with 32-bit
    byte offsets and 2^31 as the out-of-range sentinel, so a stage whose
    half-tensor reaches 2^31 bytes is refused at creation (PETRA_ERR_SHAPE);
    one just below is accepted.  Host only: creation allocates nothing."""
    from paper_2406_02052_amd import _lib as L
    wl = synth.CIFAR_STAGE            # 32 x 32 x 32 bf16: 65536 bytes per image
    per_image = wl.h * wl.w * wl.c_half * 2
    limit_n = (1 << 31) // per_image  # first batch at the limit
    d = _desc(wl)
    d.n = limit_n
    with pytest.raises(L.PetraError) as e:
        L.petra_stage_create(d)
    assert e.value.name == "PETRA_ERR_SHAPE"
    assert "2^31" in L.petra_last_error()
    d.n = limit_n - 1
    h = L.petra_stage_create(d)
    L.petra_stage_destroy(h)


def test_bind_and_call_validation_without_device_work():
    from paper_2406_02052_amd import _lib as L
    wl = synth.CIFAR_STAGE.with_(n=2, h=4, w=4)
    h = L.petra_stage_create(_desc(wl))
    try:
        _, _, _, ws = L.petra_stage_query(h)
        base = 1 << 40   # fake, aligned device addresses; nothing is dereferenced
        with pytest.raises(L.PetraError) as e:
            L.petra_stage_forward(h, base, base + 4096, base + 8192, base + 12288, 0)
        assert e.value.name == "PETRA_ERR_STATE"
        with pytest.raises(L.PetraError) as e:
            L.petra_stage_bind(h, base, base, base, base, base, base, ws - 1)
        assert e.value.name == "PETRA_ERR_WORKSPACE"
        with pytest.raises(L.PetraError) as e:
            L.petra_stage_bind(h, base + 4, base, base, base, base, base, ws)
        assert e.value.name == "PETRA_ERR_ALIGN"
        L.petra_stage_bind(h, base, base, base, base, base, base + (1 << 30), ws)
        n = wl.n * wl.h * wl.w * wl.c_half * 2
        x1, x2, y1, y2 = (base + (2 << 30) + i * 65536 for i in range(4))
        with pytest.raises(L.PetraError) as e:     # y1 half-overlaps x1
            L.petra_stage_forward(h, x1, x2, x1 + 16, y2, 0)
        assert e.value.name == "PETRA_ERR_ALIAS"
        with pytest.raises(L.PetraError) as e:     # misaligned activation
            L.petra_stage_forward(h, x1 + 8, x2, y1, y2, 0)
        assert e.value.name == "PETRA_ERR_ALIGN"
        with pytest.raises(L.PetraError) as e:     # dx1 overlaps y2
            L.petra_stage_reconstruct_backward(h, y1, y2, x1, x2, base + (3 << 30), base + (4 << 30),
                                               y2, base + (5 << 30), 0)
        assert e.value.name == "PETRA_ERR_ALIAS"
        with pytest.raises(L.PetraError) as e:
            L.petra_stage_set_optimizer(h, L.Sgd(0.1, 1.0, 0.0, 1, 1))
        assert e.value.name == "PETRA_ERR_INVALID_ARG"
        with pytest.raises(L.PetraError) as e:
            L.petra_stage_set_optimizer(h, L.Sgd(0.1, 0.9, 0.0, 1, 0))
        assert e.value.name == "PETRA_ERR_INVALID_ARG"
        assert n > 0
    finally:
        L.petra_stage_destroy(h)


def test_net_backprop_step_validation_without_device_work():
    from paper_2406_02052_amd import _lib as L
    from paper_2406_02052_amd.stage import ctypes_int_array
    wl = synth.REVNET18_SCHEDULE.with_(n=2, h=8, w=8, widths=(16, 32), blocks_per_stage=1)
    desc = L.NetDesc(wl.n, wl.h, wl.w, wl.c_img, len(wl.widths), ctypes_int_array(wl.widths),
                     wl.blocks_per_stage, wl.classes, L.PETRA_FP32, wl.bn_eps, wl.bn_momentum)
    h = L.petra_net_create(desc)
    try:
        _, _, _, ws = L.petra_net_query(h)
        base = 1 << 40   # fake, aligned device addresses; nothing is dereferenced
        img, lab = base + (2 << 30), base + (3 << 30)
        with pytest.raises(L.PetraError) as e:
            L.petra_net_backprop_step(h, img, lab, None, 0)
        assert e.value.name == "PETRA_ERR_STATE"
        L.petra_net_bind(h, base, base, base, base, base, base + (1 << 30), ws)
        with pytest.raises(L.PetraError) as e:
            L.petra_net_backprop_step(h, None, lab, None, 0)
        assert e.value.name == "PETRA_ERR_INVALID_ARG"
        with pytest.raises(L.PetraError) as e:
            L.petra_net_backprop_step(h, img + 8, lab, None, 0)
        assert e.value.name == "PETRA_ERR_ALIGN"
        with pytest.raises(L.PetraError) as e:
            L.petra_net_backprop_step(h, img, lab, base + (4 << 30) + 4, 0)
        assert e.value.name == "PETRA_ERR_ALIGN"
    finally:
        L.petra_net_destroy(h)


def test_net_split_stage_layout_and_validation():
    """Per-layer split: same parameters in the same canonical order, one stage
    per front layer and per block; bad flags are rejected."""
    from paper_2406_02052_amd import _lib as L
    from paper_2406_02052_amd.stage import ctypes_int_array
    wl = synth.REVNET18_SCHEDULE
    def desc(split, ib=0):
        return L.NetDesc(wl.n, wl.h, wl.w, wl.c_img, len(wl.widths), ctypes_int_array(wl.widths),
                         wl.blocks_per_stage, wl.classes, L.PETRA_BF16, wl.bn_eps, wl.bn_momentum,
                         ib, 0, split)
    infos = {}
    for split in (0, 1):
        h = L.petra_net_create(desc(split))
        try:
            n_params, nt, nbn, _ = L.petra_net_query(h)
            J = L.petra_net_num_stages(h)
            assert J == (len(wl.widths) * (1 + wl.blocks_per_stage) if split else len(wl.widths))
            spans = [L.petra_net_stage_params(h, j) for j in range(J)]
            assert spans[0][0] == 0 and sum(n for _, n in spans) == n_params
            assert all(a[0] + a[1] == b[0] for a, b in zip(spans, spans[1:]))
            infos[split] = [(L.petra_net_param_info(h, i).numel,
                             tuple(L.petra_net_param_info(h, i).shape)) for i in range(nt)]
        finally:
            L.petra_net_destroy(h)
    assert infos[0] == infos[1]
    with pytest.raises(L.PetraError) as e:
        L.petra_net_create(desc(2))
    assert e.value.name == "PETRA_ERR_INVALID_ARG"
