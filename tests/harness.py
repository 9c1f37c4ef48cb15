"""Test-side helpers: drive a stage through the C ABI and the oracle on the
same seeded inputs, and compare.  (Test infrastructure; not product code.)"""
from __future__ import annotations

import numpy as np

import synth
from oracle.stage import StageState


def rel(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    nb = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / nb) if nb > 0 else float(np.linalg.norm(a))


def tol(wl) -> float:
    return 1e-4 if wl.dtype == "fp32" else 2e-2


def oracle_state(wl, params, storage=True) -> StageState:
    """Oracle of the workload.  For bf16 workloads the weights are read through
    their bf16 compute copy and, when `storage` is set, activations and
    activation gradients are held at bf16 where the method materialises them
    (so ReLU decisions are taken on the stored values); storage=False gives the
    plain fp64 reference."""
    names = [n for n, _ in wl.param_shapes()]
    bf = wl.dtype == "bf16"
    return StageState(params, names, 2 if wl.kind == "basic" else 3, eps=wl.bn_eps,
                      bn_momentum=wl.bn_momentum, weight_view=synth.round_bf16 if bf else None,
                      store=synth.round_bf16 if (bf and storage) else None)


def gpu_stage(wl, params, device="cuda"):
    from paper_2406_02052_amd import Stage
    st = Stage(wl.n, wl.h, wl.w, wl.c_half, wl.blocks, wl.kind, wl.dtype, c_mid=wl.c_mid,
               bn_eps=wl.bn_eps, bn_momentum=wl.bn_momentum, device=device)
    st.set_params(params)
    st.set_optimizer(lr=wl.lr, momentum=wl.momentum, weight_decay=wl.weight_decay,
                     nesterov=wl.nesterov, accum_k=wl.accum_k)
    return st


def run_step_parity(wl, bn_affine="random", check_update=True):
    """Forward, reconstruct+VJP and update on both sides; returns an error dict."""
    import torch
    from paper_2406_02052_amd import to_host

    params = synth.stage_params(wl, bn_affine)
    ref = oracle_state(wl, params)
    exact = oracle_state(wl, params, storage=False) if wl.dtype == "bf16" else None
    st = gpu_stage(wl, params)
    x1, x2 = synth.stage_input(wl)
    g1, g2 = synth.stage_output_grad(wl)
    errs = {}
    # forward
    y1, y2 = st.act(), st.act()
    st.forward(st.act(x1), st.act(x2), y1, y2)
    oy1, oy2 = ref.forward(x1, x2)
    torch.cuda.synchronize()
    errs["y1"] = rel(to_host(y1), oy1)
    errs["y2"] = rel(to_host(y2), oy2)
    # backward from the oracle output in storage precision (same bits on both sides)
    yin1, yin2 = synth.to_storage(oy1, wl.dtype), synth.to_storage(oy2, wl.dtype)
    p0 = st.get_params()
    rx1, rx2, dx1, dx2 = st.act(), st.act(), st.act(), st.act()
    st.reconstruct_backward(st.act(yin1), st.act(yin2), st.act(g1), st.act(g2), rx1, rx2, dx1, dx2)
    ox1, ox2, odx1, odx2, ograds = ref.backward(yin1, yin2, g1, g2, k=wl.accum_k)
    torch.cuda.synchronize()
    errs["x1"] = rel(to_host(rx1), ox1)
    errs["x2"] = rel(to_host(rx2), ox2)
    errs["dx1"] = rel(to_host(dx1), odx1)
    errs["dx2"] = rel(to_host(dx2), odx2)
    errs["drift_gpu"] = max(rel(to_host(rx1), x1), rel(to_host(rx2), x2))
    errs["drift_oracle"] = max(rel(ox1, x1), rel(ox2, x2))
    if exact is not None:
        # informational: distance of the bf16 path from plain fp64 arithmetic
        ex = exact.backward(yin1, yin2, g1, g2, k=wl.accum_k)
        errs["fp64_dx"] = max(rel(to_host(dx1), ex[2]), rel(to_host(dx2), ex[3]))
    grads = st.get_grads()
    names = [n for n, _ in wl.param_shapes()]
    gerr = {}
    for nm, g, og in zip(names, grads, ref.accum):
        gerr[nm] = rel(g, og)
    errs["grad_max"] = max(gerr.values())
    errs["grad_worst"] = max(gerr, key=gerr.get)
    rm, rv = st.run_mean.cpu().numpy(), st.run_var.cpu().numpy()
    orm = np.concatenate([m.reshape(-1) for m in ref.run_mean])
    orv = np.concatenate([v.reshape(-1) for v in ref.run_var])
    errs["run_mean"] = rel(rm, orm)
    errs["run_var"] = rel(rv, orv)
    if check_update:
        st.update()
        ref.update(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
        torch.cuda.synchronize()
        p1 = st.get_params()
        inc = [rel(a - b, np.asarray(c) - np.asarray(pb, np.float64))
               for a, b, c, pb in zip(p1, p0, ref.params, params)]
        errs["update_inc"] = max(inc)
        mom = st.get_momentum()
        errs["momentum"] = max(rel(a, b) for a, b in zip(mom, ref.buf))
        errs["accum_zero"] = float(max(np.abs(g).max() for g in st.get_grads()))
    return errs


def assert_errs(errs, wl):
    t = tol(wl)
    bad = {k: v for k, v in errs.items()
           if k not in ("drift_gpu", "drift_oracle", "grad_worst", "accum_zero", "fp64_dx")
           and not v <= t}
    assert not bad, f"parity failed (tol {t}): {bad}\nall: {errs}"
    assert errs.get("accum_zero", 0.0) == 0.0
