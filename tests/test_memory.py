"""Memory accounting (Tables 3 and 6): the library's per-stage plan against the
definition of the buffers (one copy per micro-batch in flight), and the
host-side estimate's structure.  Host only: no device memory is allocated."""
import numpy as np
import pytest

import synth


def _net(wl, ib, pb):
    from paper_2406_02052_amd import _lib as L
    from paper_2406_02052_amd.stage import ctypes_int_array
    desc = L.NetDesc(wl.n, wl.h, wl.w, wl.c_img, len(wl.widths), ctypes_int_array(wl.widths),
                     wl.blocks_per_stage, wl.classes,
                     L.PETRA_BF16 if wl.dtype == "bf16" else L.PETRA_FP32, wl.bn_eps,
                     wl.bn_momentum, int(ib), int(pb))
    return L, L.petra_net_create(desc)


def _align(v):
    return (v + 255) // 256 * 256


@pytest.mark.parametrize("ib,pb", [(False, False), (True, False), (False, True), (True, True)])
def test_library_plan_matches_buffer_definitions(ib, pb):
    wl = synth.REVNET18_SCHEDULE
    L, h = _net(wl, ib, pb)
    try:
        n_params, _, n_bn, ws = L.petra_net_query(h)
        J = len(wl.widths)
        esz = 2 if wl.dtype == "bf16" else 4
        rows = [L.petra_net_memory(h, j) for j in range(J)]
        spans = [L.petra_net_stage_params(h, j) for j in range(J)]
        assert sum(n for _, n in spans) == n_params
        # the workspace parts add up to the queried workspace exactly
        assert sum(r["total"] - r["params"] for r in rows) == ws
        assert sum(r["params"] for r in rows) == 3 * 4 * n_params + 2 * 4 * n_bn
        for j, r in enumerate(rows):
            inflight = 2 * (J - 1 - j) + 1
            m = wl.n * (wl.h >> j) * (wl.w >> j)
            last = j == J - 1
            assert r["input_buffer"] == (inflight * _align(m * wl.widths[j] * esz)
                                         if ib and not last else 0)
            if pb and not last:
                # one fp32 copy of the stage's parameters per micro-batch in
                # flight, plus the compute copies of its conv weights
                assert r["param_buffer"] >= inflight * 4 * spans[j][1]
                assert r["param_buffer"] <= inflight * (4 + 3 * esz) * spans[j][1] + inflight * 5 * 256
            else:
                assert r["param_buffer"] == 0
            assert r["activation_buffer"] > 0 and r["weight_copies"] > 0 and r["scratch"] > 0
    finally:
        L.petra_net_destroy(h)


def test_buffers_only_add_their_own_bytes():
    wl = synth.REVNET18_SCHEDULE
    J = len(wl.widths)
    tab = {}
    for ib in (False, True):
        for pb in (False, True):
            L, h = _net(wl, ib, pb)
            tab[(ib, pb)] = [L.petra_net_memory(h, j) for j in range(J)]
            L.petra_net_destroy(h)
    base = tab[(False, False)]
    for key, rows in tab.items():
        for r, b in zip(rows, base):
            for field in ("params", "weight_copies", "activation_buffer"):
                assert r[field] == b[field], (key, field)
    # PETRA (neither buffer) is the smallest; the input buffer costs more than the stash
    tot = {k: sum(r["total"] for r in v) for k, v in tab.items()}
    assert tot[(False, False)] < tot[(False, True)] < tot[(True, False)] < tot[(True, True)]


def test_estimate_structure_revnet50():
    from paper_2406_02052_amd import memory as M
    stages = M.revnet50_imagenet_18(64)
    assert len(stages) == 18
    assert [s.kind for s in stages].count("nonrev") == 5      # stem, 3 downsamplings, head
    rows = {(ib, pb): M.estimate(stages, ib, pb) for ib in (False, True) for pb in (False, True)}
    J = 18
    for (ib, pb), rs in rows.items():
        for j, (s, r) in enumerate(zip(stages, rs)):
            k = 2 * (J - 1 - j) + 1
            assert r["param_buffer"] == (k * 4 * s.params if pb else 0)
            assert r["input_buffer"] == (k * 4 * s.in_elems if ib and s.kind == "rev" else 0)
            assert r["activation_buffer"] == (k * 4 * s.in_elems if s.kind == "nonrev" else 0)
    tab = M.savings_table(stages)
    assert tab[0]["saving_pct"] == 0.0
    assert 0 < tab[1]["saving_pct"] < tab[2]["saving_pct"] < tab[3]["saving_pct"] < 100
