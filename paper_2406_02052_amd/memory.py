"""Memory accounting of the schedule's buffers (Table 3 and Table 6 analogs).

Two sources:

* `net_memory(net)`: the device bytes the library's one-GPU schedule actually
  plans, per stage and by purpose (`petra_net_memory`), for a `Net` built with
  or without the input and parameter buffers.
* `estimate(...)`: a host-side model for networks the library does not build,
  e.g. the 18-stage RevNet-50 on ImageNet at batch 64 the paper's Table 3
  estimates.  Stage j of J (0-based) holds 2(J-1-j) + 1 micro-batches between
  their forward and their backward (the delay of the method's analysis plus
  the one being processed); a non-reversible stage always keeps its input for
  each of them, a reversible stage only with the input buffer; the parameter
  buffer keeps one fp32 copy of the stage's parameters for each.  Every stage
  also holds its fp32 parameters, gradient accumulator and momentum and one
  micro-batch's working set.
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List

from . import _lib as L


def net_memory(net) -> List[Dict[str, int]]:
    """Per-stage byte counts of an instantiated Net (see petra_net_mem)."""
    return [L.petra_net_memory(net.handle, j) for j in range(net.n_stages)]


@dataclasses.dataclass(frozen=True)
class StageShape:
    kind: str          # "nonrev" (stem, downsampling, head) or "rev" (reversible blocks)
    in_elems: int      # elements of the stage's input, one micro-batch
    params: int        # parameter count
    work_elems: int    # activation elements of one micro-batch's working set


def _rev_bottleneck(n, h, w, c, mid, blocks=1) -> StageShape:
    half = c // 2
    per_fn = half * mid + 9 * mid * mid + mid * half + 2 * (mid + mid + half)
    hw = n * h * w
    # input, output, and the three pre-BN tensors of the function being rebuilt
    return StageShape("rev", hw * c, 2 * blocks * per_fn, hw * (2 * c + mid + mid + half))


def revnet50_imagenet_18(n: int = 64) -> List[StageShape]:
    """Reading of an 18-stage RevNet-50 split on 224x224 ImageNet, following the
    grouping of the 18-stage split in Table 6 (stem | 4 reversible | downsampling
    | 3 | downsampling | 3 | downsampling | 3 | head): bottleneck blocks of width
    256, 512, 1024, 2048 at 56, 28, 14, 7 pixels with inner width a quarter of
    the half width (two streams of c/2, as the library's bottleneck blocks);
    the stem is a 7x7 stride-2 conv to 64 channels, BN, ReLU, 3x3 max-pool and a
    1x1 conv to 256; each downsampling is a 1x1 stride-2 conv doubling the
    width, with BN; the head pools and applies a 2048 x 1000 linear layer."""
    out = [StageShape("nonrev", n * 224 * 224 * 3, 7 * 7 * 3 * 64 + 2 * 64 + 64 * 256 + 2 * 256,
                      n * (112 * 112 * 64 * 2 + 56 * 56 * 64 + 56 * 56 * 256 * 2))]
    res, c = 56, 256
    for level, count in enumerate((4, 3, 3, 3)):
        if level > 0:
            out.append(StageShape("nonrev", n * res * res * c, c * 2 * c + 2 * 2 * c,
                                  n * (res * res * c + 2 * (res // 2) ** 2 * 2 * c)))
            res, c = res // 2, 2 * c
        out += [_rev_bottleneck(n, res, res, c, c // 8) for _ in range(count)]
    out.append(StageShape("nonrev", n * res * res * c, c * 1000 + 1000, n * (res * res * c + c)))
    return out


def estimate(stages: List[StageShape], input_buffer: bool, param_buffer: bool,
             act_bytes: int = 4) -> List[Dict[str, int]]:
    """Per-stage bytes of the model described in the module notes."""
    J = len(stages)
    rows = []
    for j, s in enumerate(stages):
        inflight = 2 * (J - 1 - j) + 1
        r = {"params": 3 * 4 * s.params,
             "activation_buffer": inflight * s.in_elems * act_bytes if s.kind == "nonrev" else 0,
             "input_buffer": inflight * s.in_elems * act_bytes
             if (s.kind == "rev" and input_buffer) else 0,
             "param_buffer": inflight * 4 * s.params if param_buffer else 0,
             "scratch": s.work_elems * act_bytes}
        r["total"] = sum(r.values())
        rows.append(r)
    return rows


def savings_table(stages: List[StageShape], act_bytes: int = 4) -> List[Dict[str, float]]:
    """Table 3 layout: total bytes for the four buffer settings and the saving
    relative to keeping both."""
    out = []
    base = None
    for ib, pb in ((True, True), (True, False), (False, True), (False, False)):
        tot = sum(r["total"] for r in estimate(stages, ib, pb, act_bytes))
        base = tot if base is None else base
        out.append({"input_buffer": ib, "param_buffer": pb, "bytes": tot,
                    "saving_pct": 100.0 * (1.0 - tot / base)})
    return out
