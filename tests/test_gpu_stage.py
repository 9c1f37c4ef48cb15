"""GPU parity of the reversible stage step against the oracle (through the C ABI)."""
import numpy as np
import pytest

import synth
from tests.harness import assert_errs, run_step_parity

pytestmark = pytest.mark.gpu

SMALL = {
    # exact workload of the fp32 single-block case
    "fp32_block_8x8x8x32": synth.BLOCK_FP32,
    # one partial tile, ragged reduction (K = 144), two blocks
    "fp32_ragged_3x7x5_c16": synth.BLOCK_FP32.with_(n=3, h=7, w=5, blocks=2),
    "fp32_3tiles_5x9x7_c32": synth.BLOCK_FP32.with_(n=5, h=9, w=7, c_half=32, blocks=1),
    "fp32_bottleneck_2x6x6": synth.BLOCK_FP32.with_(n=2, h=6, w=6, c_half=32, c_mid=16,
                                                     kind="bottleneck", blocks=1),
    "bf16_c32_4x9x9": synth.CIFAR_STAGE.with_(n=4, h=9, w=9),
    "bf16_c64_2x10x10": synth.CIFAR_STAGE.with_(n=2, h=10, w=10, c_half=64, blocks=1),
    "bf16_c128_3x6x6": synth.IMAGENET32_STAGE.with_(n=3, h=6, w=6, blocks=2),
    "bf16_bottleneck_2x12x12": synth.IMAGENET_BOTTLENECK_STAGE.with_(n=2, h=12, w=12, blocks=2),
}


@pytest.mark.parametrize("name", list(SMALL))
def test_stage_step_parity_small(name):
    wl = SMALL[name]
    print(f"case {name}: {wl}", flush=True)
    errs = run_step_parity(wl, bn_affine="random")
    print(name, errs, flush=True)
    assert_errs(errs, wl)


def test_config_fp32_block_identity_bn():
    wl = synth.BLOCK_FP32
    errs = run_step_parity(wl, bn_affine="identity")
    print(errs, flush=True)
    assert_errs(errs, wl)
