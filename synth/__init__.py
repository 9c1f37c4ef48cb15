"""Seeded synthetic workloads shared by the oracle-side tests and the HIP side.

This module holds *no* arithmetic of the method: it only names the workload
shapes, draws seeded random tensors, and rounds fp32 values to bf16 so that
both sides receive bit-identical inputs.  Nothing here convolves, normalises
or differentiates anything.

Seeds: numpy ``default_rng(2406 + i)`` with i = 0 for the stage input,
i = 1 for the output gradient, i = 2 + p for the p-th parameter tensor in
canonical order, i = 99 for class labels.  Values are drawn in fp32; for the
bf16 workloads they are rounded to nearest-even bf16 (values stay fp32 arrays
whose bit patterns are exactly representable in bf16).
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, List, Tuple

import numpy as np

SEED_BASE = 2406


@dataclasses.dataclass(frozen=True)
class StageWorkload:
    """One reversible stage at a fixed shape (activations are NHWC)."""
    name: str
    dtype: str            # "fp32" or "bf16" (storage); accumulation is fp32
    n: int
    h: int
    w: int
    c_half: int           # channels per stream; the full activation has 2*c_half
    kind: str             # "basic" or "bottleneck"
    blocks: int
    c_mid: int = 0        # bottleneck inner width
    x_dist: str = "normal"      # "normal" or "abs_normal"
    dy_sigma: float = 1.0
    lr: float = 0.1
    momentum: float = 0.9
    weight_decay: float = 0.0
    nesterov: bool = True
    accum_k: int = 1
    bn_eps: float = 1e-5
    bn_momentum: float = 0.1

    @property
    def images(self) -> int:
        return self.n

    def conv_layers(self) -> List[Tuple[int, int, int, int]]:
        """(C_out, R, S, C_in) of each conv of one residual function."""
        c = self.c_half
        if self.kind == "basic":
            return [(c, 3, 3, c), (c, 3, 3, c)]
        m = self.c_mid
        return [(m, 1, 1, c), (m, 3, 3, m), (c, 1, 1, m)]

    def param_shapes(self) -> List[Tuple[str, Tuple[int, ...]]]:
        """Canonical parameter order: block b, function F then G, conv l:
        weight [C_out,R,S,C_in] (KRSC), BN gamma [C_out], BN beta [C_out]."""
        out = []
        for b in range(self.blocks):
            for f in ("F", "G"):
                for l, (co, r, s, ci) in enumerate(self.conv_layers()):
                    out.append((f"b{b}.{f}.conv{l}.weight", (co, r, s, ci)))
                    out.append((f"b{b}.{f}.bn{l}.gamma", (co,)))
                    out.append((f"b{b}.{f}.bn{l}.beta", (co,)))
        return out

    def with_(self, **kw) -> "StageWorkload":
        return dataclasses.replace(self, **kw)


# The five workloads of the build, named by what they are.
BLOCK_FP32 = StageWorkload("block_fp32_8x8x8x32", "fp32", 8, 8, 8, 16, "basic", 1,
                           x_dist="normal", dy_sigma=1.0)
CIFAR_STAGE = StageWorkload("cifar_revnet18_stage_128x32x32x64", "bf16", 128, 32, 32, 32,
                            "basic", 2, x_dist="normal", dy_sigma=1e-2)
IMAGENET32_STAGE = StageWorkload("imagenet32_revnet34_stage_256x16x16x256", "bf16", 256, 16,
                                 16, 128, "basic", 6, x_dist="abs_normal", dy_sigma=1e-3)
IMAGENET_BOTTLENECK_STAGE = StageWorkload("imagenet_revnet50_bottleneck_stage_64x56x56x256",
                                          "bf16", 64, 56, 56, 128, "bottleneck", 3, c_mid=32,
                                          x_dist="abs_normal", dy_sigma=1e-3)

STAGE_WORKLOADS: Dict[str, StageWorkload] = {
    w.name: w for w in (BLOCK_FP32, CIFAR_STAGE, IMAGENET32_STAGE, IMAGENET_BOTTLENECK_STAGE)
}


@dataclasses.dataclass(frozen=True)
class NetWorkload:
    """RevNet-18-shaped network split into J stages (CIFAR-shaped images)."""
    name: str = "revnet18_petra_schedule_128x32x32x3"
    dtype: str = "bf16"
    n: int = 128
    h: int = 32
    w: int = 32
    c_img: int = 3
    widths: Tuple[int, ...] = (64, 128, 256, 512)   # full width (both streams) per stage
    blocks_per_stage: int = 2
    classes: int = 10
    ticks: int = 100
    lr: float = 0.1
    momentum: float = 0.9
    weight_decay: float = 5e-4
    nesterov: bool = True
    accum_k: int = 1
    bn_eps: float = 1e-5
    bn_momentum: float = 0.1

    @property
    def stages(self) -> int:
        return len(self.widths)

    def with_(self, **kw) -> "NetWorkload":
        return dataclasses.replace(self, **kw)


REVNET18_SCHEDULE = NetWorkload()


# ---------------------------------------------------------------------------
# bf16 rounding (input preparation only)
# ---------------------------------------------------------------------------

def round_bf16(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).reshape(a.shape)


def to_storage(a: np.ndarray, dtype: str) -> np.ndarray:
    a = np.asarray(a, dtype=np.float32)
    return round_bf16(a) if dtype == "bf16" else np.ascontiguousarray(a)


def rng(i: int) -> np.random.Generator:
    return np.random.default_rng(SEED_BASE + i)


def he_std(shape: Tuple[int, ...]) -> float:
    """He-normal standard deviation for a KRSC weight: sqrt(2 / (R*S*C_in))."""
    _, r, s, ci = shape
    return math.sqrt(2.0 / (r * s * ci))


# ---------------------------------------------------------------------------
# Stage inputs
# ---------------------------------------------------------------------------

def stage_input(wl: StageWorkload, seed_offset: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    """x = [x1 | x2] of shape [N,H,W,2*C/2]; returns the two contiguous halves."""
    shape = (wl.n, wl.h, wl.w, 2 * wl.c_half)
    x = rng(0 + seed_offset).standard_normal(shape, dtype=np.float32)
    if wl.x_dist == "abs_normal":
        x = np.abs(x)
    x = to_storage(x, wl.dtype)
    c = wl.c_half
    return np.ascontiguousarray(x[..., :c]), np.ascontiguousarray(x[..., c:])


def stage_output_grad(wl: StageWorkload, seed_offset: int = 0) -> Tuple[np.ndarray, np.ndarray]:
    shape = (wl.n, wl.h, wl.w, 2 * wl.c_half)
    g = rng(1 + seed_offset).standard_normal(shape, dtype=np.float32) * np.float32(wl.dy_sigma)
    g = to_storage(g, wl.dtype)
    c = wl.c_half
    return np.ascontiguousarray(g[..., :c]), np.ascontiguousarray(g[..., c:])


def stage_params(wl: StageWorkload, bn_affine: str = "identity") -> List[np.ndarray]:
    """Parameters in canonical order (fp32 arrays; conv weights rounded to the
    storage dtype so both sides start from the same values).

    bn_affine: "identity" gives gamma=1, beta=0; "random" draws gamma in
    [0.5, 1.5) and beta ~ N(0, 0.2) (used by tests so the affine terms matter).
    """
    out = []
    for p, (name, shape) in enumerate(wl.param_shapes()):
        g = rng(2 + p)
        if name.endswith("weight"):
            v = g.standard_normal(shape, dtype=np.float32) * np.float32(he_std(shape))
            v = to_storage(v, wl.dtype)
        elif name.endswith("gamma"):
            v = (np.ones(shape, np.float32) if bn_affine == "identity"
                 else (0.5 + g.random(shape, dtype=np.float32)).astype(np.float32))
        else:
            v = (np.zeros(shape, np.float32) if bn_affine == "identity"
                 else (0.2 * g.standard_normal(shape, dtype=np.float32)).astype(np.float32))
        out.append(np.ascontiguousarray(v))
    return out


def is_weight_decayed(name: str) -> bool:
    """Weight decay applies to conv / FC weights only, never to BN parameters
    or biases (Sec. 4.1, experimental setup)."""
    return name.endswith("weight")


# ---------------------------------------------------------------------------
# Network (multi-stage schedule) inputs
# ---------------------------------------------------------------------------

def net_param_shapes(wl: NetWorkload) -> List[Tuple[str, Tuple[int, ...]]]:
    """Canonical parameter order of the J-stage network.

    stage 0: stem conv3x3 (c_img -> widths[0]) + BN, then the reversible blocks.
    stage j>0: transition conv1x1 stride 2 (widths[j-1] -> widths[j]) + BN,
    then the reversible blocks.  The last stage also owns the FC head.
    """
    out = []
    for j, wdt in enumerate(wl.widths):
        if j == 0:
            out.append((f"s{j}.stem.weight", (wdt, 3, 3, wl.c_img)))
        else:
            out.append((f"s{j}.trans.weight", (wdt, 1, 1, wl.widths[j - 1])))
        pre = "stem" if j == 0 else "trans"
        out.append((f"s{j}.{pre}_bn.gamma", (wdt,)))
        out.append((f"s{j}.{pre}_bn.beta", (wdt,)))
        c = wdt // 2
        for b in range(wl.blocks_per_stage):
            for f in ("F", "G"):
                for l in range(2):
                    out.append((f"s{j}.b{b}.{f}.conv{l}.weight", (c, 3, 3, c)))
                    out.append((f"s{j}.b{b}.{f}.bn{l}.gamma", (c,)))
                    out.append((f"s{j}.b{b}.{f}.bn{l}.beta", (c,)))
    out.append((f"s{len(wl.widths) - 1}.fc.weight", (wl.classes, wl.widths[-1])))
    out.append((f"s{len(wl.widths) - 1}.fc.bias", (wl.classes,)))
    return out


def net_params(wl: NetWorkload) -> List[np.ndarray]:
    out = []
    for p, (name, shape) in enumerate(net_param_shapes(wl)):
        g = rng(2 + p)
        if name.endswith("fc.weight"):
            v = g.standard_normal(shape, dtype=np.float32) * np.float32(math.sqrt(2.0 / shape[1]))
            v = to_storage(v, wl.dtype)
        elif name.endswith("weight"):
            v = g.standard_normal(shape, dtype=np.float32) * np.float32(he_std(shape))
            v = to_storage(v, wl.dtype)
        elif name.endswith("gamma"):
            v = np.ones(shape, np.float32)
        else:  # beta, bias
            v = np.zeros(shape, np.float32)
        out.append(np.ascontiguousarray(v))
    return out


def net_images(wl: NetWorkload, count: int) -> np.ndarray:
    """`count` micro-batches of N(0,1) images, [count, N, H, W, c_img]."""
    x = rng(0).standard_normal((count, wl.n, wl.h, wl.w, wl.c_img), dtype=np.float32)
    return to_storage(x, wl.dtype)


def net_labels(wl: NetWorkload, count: int) -> np.ndarray:
    return rng(99).integers(0, wl.classes, size=(count, wl.n), dtype=np.int32)
