"""GPU parity of the one-GPU multi-stage PETRA schedule against the oracle's
tick simulator (Alg. 1, Eq. 5, delays 2(J - j))."""
import numpy as np
import pytest

import synth
from oracle.net import PetraNet
from tests.harness import CHAIN_COS, CHAIN_TOL, TOL, cos_sim, rel

pytestmark = pytest.mark.gpu

# Four stages down to 2x2 pixels: every BN normalises at least 16 rows (with a
# handful of rows the BN gain 1/sqrt(var + eps) amplifies rounding without
# bound and the comparison stops measuring the kernels); lr 0.02 keeps the
# short trajectory out of the exploding regime.
TINY = synth.REVNET18_SCHEDULE.with_(n=4, h=16, w=16, widths=(16, 32, 64, 128), blocks_per_stage=1,
                                     lr=0.02)


def affine_params(wl, seed=12):
    names = [n for n, _ in synth.net_param_shapes(wl)]
    params = synth.net_params(wl)
    rng = np.random.default_rng(seed)
    for i, nm in enumerate(names):
        if nm.endswith("gamma"):
            params[i] = (0.8 + 0.4 * rng.random(params[i].shape)).astype(np.float32)
        elif nm.endswith("beta") or nm.endswith("bias"):
            params[i] = (0.1 * rng.standard_normal(params[i].shape)).astype(np.float32)
    return names, params


def run_both(wl, names, params, n_micro, ticks, store=None, gpu=True, mode=0, split=False):
    import torch
    from paper_2406_02052_amd import Net

    rng = np.random.default_rng(3)
    imgs = [synth.to_storage(rng.standard_normal((wl.n, wl.h, wl.w, wl.c_img), dtype=np.float32),
                             wl.dtype) for _ in range(n_micro)]
    labs = [rng.integers(0, wl.classes, wl.n).astype(np.int32) for _ in range(n_micro)]
    bf = wl.dtype == "bf16"
    ref = PetraNet([p.astype(np.float64) for p in params], names, len(wl.widths),
                   wl.blocks_per_stage, weight_view=synth.round_bf16 if bf else None,
                   store=store if store is not None else (synth.round_bf16 if bf else None),
                   use_inputs=bool(mode & 1), use_params=bool(mode & 2), split_fronts=split)
    oloss = []
    for t in range(ticks):
        oloss.append(ref.tick(t, lambda m: imgs[m], lambda m: labs[m], n_micro, wl.lr,
                              wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k))
    if not gpu:
        return ref, oloss, None, None
    net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype,
              input_buffer=bool(mode & 1), param_buffer=bool(mode & 2), split_stages=split)
    assert net.n_stages == ref.J
    net.set_params(params)
    net.set_optimizer(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
    gloss = []
    for t in range(ticks):
        if t < n_micro:
            wrote = net.tick(net.images(imgs[t]), net.labels(labs[t]))
        else:
            wrote = net.tick()
        torch.cuda.synchronize()
        gloss.append(float(net.loss.item()) if wrote else None)
    return ref, oloss, net, gloss


def compare(wl, names, params, ref, oloss, net, gloss, tol_loss, tol_param, tol_stats=None):
    assert [l is None for l in oloss] == [l is None for l in gloss], (oloss, gloss)
    for a, b in zip(gloss, oloss):
        if b is not None:
            assert abs(a - b) <= tol_loss * abs(b), (a, b)
    got = dict(zip(names, net.get_params()))
    want = {}
    for st in ref.stages:
        for nm, p in zip(st.names, st.params):
            want[nm] = p
    p0 = dict(zip(names, params))
    # Some increments vanish identically (a stage's last BN beta feeding a BN'd
    # downsampling sees a shift-invariant loss): errors are taken relative to
    # max(|increment|, 1e-3 |all increments|).
    total = np.sqrt(sum(float(np.sum((np.asarray(want[nm]) - p0[nm]) ** 2)) for nm in names))
    worst = (0.0, "")
    for nm in names:
        d_ref = np.asarray(want[nm], np.float64) - p0[nm]
        d_got = np.asarray(got[nm], np.float64) - p0[nm]
        e = float(np.linalg.norm(d_got - d_ref) / max(np.linalg.norm(d_ref), 1e-3 * total))
        assert e <= tol_param, (nm, e, tol_param)
        worst = max(worst, (e, nm))
    # the net's running statistics are laid out per stage as [front, blocks...]
    orm = np.concatenate([np.concatenate([m.reshape(-1) for m in st.run_mean]) for st in ref.stages])
    orv = np.concatenate([np.concatenate([v.reshape(-1) for v in st.run_var]) for st in ref.stages])
    ts = tol_loss if tol_stats is None else tol_stats
    for a, b in ((net.run_mean.cpu().numpy(), orm), (net.run_var.cpu().numpy(), orv)):
        assert a.shape == b.shape
        assert rel(a, b) <= ts, ("running statistics", rel(a, b), ts)
    return worst


def test_tiny_net_fp32_matches_oracle_ticks():
    wl = TINY.with_(dtype="fp32")
    names, params = affine_params(wl)
    J = len(wl.widths)
    n_micro, ticks = 3, 3 + 2 * J
    ref, oloss, net, gloss = run_both(wl, names, params, n_micro, ticks)
    print("losses", gloss, oloss, flush=True)
    worst = compare(wl, names, params, ref, oloss, net, gloss, 1e-4, 1e-4)
    print("worst parameter increment error", worst, flush=True)
    t, fed, inflight = net.state()
    assert (t, fed, inflight) == (ticks, n_micro, 0)


def test_tiny_net_bf16_matches_storage_oracle():
    """bf16 schedule against the storage-precision oracle: losses and running
    statistics (forward side) at the stated bar; the parameter increments come
    out of gradients through several reconstructed bf16 blocks and are held to
    the chain bound of tests/harness.py."""
    wl = TINY
    names, params = affine_params(wl)
    J = len(wl.widths)
    n_micro, ticks = 3, 3 + 2 * J
    ref, oloss, net, gloss = run_both(wl, names, params, n_micro, ticks)
    print("losses", gloss, oloss, flush=True)
    worst = compare(wl, names, params, ref, oloss, net, gloss, TOL["bf16"], CHAIN_TOL)
    print("worst parameter increment error", worst, flush=True)


def test_tiny_net_bf16_identity_blocks_at_stated_bar():
    """The same schedule with identity blocks (last BN of every F and G zeroed)
    and lr = 0: every backward is exact backprop through the front layers and
    the head, one function deep; momentum buffers, losses and running
    statistics at the stated bar."""
    wl = TINY.with_(lr=0.0)
    names, params = affine_params(wl)
    for i, nm in enumerate(names):
        parts = nm.split(".")
        if len(parts) == 5 and parts[3] == "bn1":
            params[i] = np.zeros_like(params[i])
    J = len(wl.widths)
    n_micro, ticks = 3, 3 + 2 * J
    ref, oloss, net, gloss = run_both(wl, names, params, n_micro, ticks)
    for a, b in zip(gloss, oloss):
        if b is not None:
            assert abs(a - b) <= TOL["bf16"] * abs(b), (a, b)
    want = {nm: np.asarray(b, np.float64) for st in ref.stages for nm, b in zip(st.names, st.buf)}
    for nm, g in zip(names, net.get_momentum()):
        if not np.any(want[nm] != 0):
            assert not np.any(g != 0), nm
        else:
            assert rel(g, want[nm]) <= TOL["bf16"], (nm, rel(g, want[nm]))


def test_full_schedule_first_losses_and_finite_run():
    """RevNet-18-shaped schedule at 128x32x32x3: the first three losses match the
    oracle's tick simulator (bf16 storage), and 40 ticks stay finite."""
    wl = synth.REVNET18_SCHEDULE
    names = [n for n, _ in synth.net_param_shapes(wl)]
    params = synth.net_params(wl)
    J = len(wl.widths)
    ref, oloss, net, gloss = run_both(wl, names, params, n_micro=J + 2, ticks=J + 2)
    print("losses", gloss, oloss, flush=True)
    for a, b in zip(gloss, oloss):
        assert (a is None) == (b is None)
        if b is not None:
            assert abs(a - b) <= 2e-2 * abs(b), (a, b)
    import torch
    rng = np.random.default_rng(5)
    t0 = net.state()[0]
    for t in range(t0, 40):
        x = synth.to_storage(rng.standard_normal((wl.n, wl.h, wl.w, wl.c_img), dtype=np.float32), "bf16")
        net.tick(net.images(x), net.labels(rng.integers(0, 10, wl.n).astype(np.int32)))
    torch.cuda.synchronize()
    assert np.isfinite(net.params.cpu().numpy()).all()
    assert np.isfinite(net.loss.item())


def run_backprop(wl, names, params, steps, store=None):
    import torch
    from paper_2406_02052_amd import Net

    rng = np.random.default_rng(4)
    imgs = [synth.to_storage(rng.standard_normal((wl.n, wl.h, wl.w, wl.c_img), dtype=np.float32),
                             wl.dtype) for _ in range(steps)]
    labs = [rng.integers(0, wl.classes, wl.n).astype(np.int32) for _ in range(steps)]
    bf = wl.dtype == "bf16"
    ref = PetraNet([p.astype(np.float64) for p in params], names, len(wl.widths),
                   wl.blocks_per_stage, weight_view=synth.round_bf16 if bf else None,
                   store=store if store is not None else (synth.round_bf16 if bf else None))
    oloss = [ref.backprop_step(imgs[i], labs[i], wl.lr, wl.momentum, wl.weight_decay,
                               wl.nesterov, wl.accum_k) for i in range(steps)]
    net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype)
    net.set_params(params)
    net.set_optimizer(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
    gloss = []
    for i in range(steps):
        net.backprop_step(net.images(imgs[i]), net.labels(labs[i]))
        torch.cuda.synchronize()
        gloss.append(float(net.loss.item()))
    return ref, oloss, net, gloss


def test_tiny_net_fp32_backprop_matches_oracle():
    """The reversible-backpropagation baseline (Table 5 comparison) against the
    oracle's sequential step: losses and parameters after three SGD steps."""
    wl = TINY.with_(dtype="fp32")
    names, params = affine_params(wl)
    ref, oloss, net, gloss = run_backprop(wl, names, params, 3)
    print("losses", gloss, oloss, flush=True)
    worst = compare(wl, names, params, ref, oloss, net, gloss, 1e-4, 1e-4)
    print("worst parameter increment error", worst, flush=True)
    orm = np.concatenate([np.concatenate([m.reshape(-1) for m in st.run_mean]) for st in ref.stages])
    np.testing.assert_allclose(net.run_mean.cpu().numpy(), orm, rtol=1e-4, atol=1e-5)
    assert net.state() == (0, 0, 0)


def test_backprop_after_drained_ticks_and_rejected_in_flight():
    import torch
    from paper_2406_02052_amd import Net, PetraError

    wl = TINY.with_(dtype="fp32")
    names, params = affine_params(wl)
    net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype)
    net.set_params(params)
    rng = np.random.default_rng(9)
    x = net.images(rng.standard_normal((wl.n, wl.h, wl.w, wl.c_img), dtype=np.float32))
    y = net.labels(rng.integers(0, wl.classes, wl.n).astype(np.int32))
    net.tick(x, y)
    with pytest.raises(PetraError) as e:
        net.backprop_step(x, y)
    assert e.value.name == "PETRA_ERR_STATE"
    J = len(wl.widths)
    for _ in range(2 * J - 2):
        net.tick()
    assert net.state()[2] == 0
    net.backprop_step(x, y)
    torch.cuda.synchronize()
    assert np.isfinite(net.loss.item())


@pytest.mark.parametrize("mode", [1, 2, 3])
def test_tiny_net_fp32_buffer_variants_match_oracle(mode):
    """Table 4 variants (input buffer, parameter buffer, both) against the
    oracle's schedule in the same variant: losses, parameters after every
    update, running statistics."""
    wl = TINY.with_(dtype="fp32")
    names, params = affine_params(wl)
    J = len(wl.widths)
    n_micro, ticks = 4, 4 + 2 * J
    ref, oloss, net, gloss = run_both(wl, names, params, n_micro, ticks, mode=mode)
    print("mode", mode, "losses", gloss, oloss, flush=True)
    worst = compare(wl, names, params, ref, oloss, net, gloss, 1e-4, 1e-4)
    print("worst parameter increment error", worst, flush=True)
    orm = np.concatenate([np.concatenate([m.reshape(-1) for m in st.run_mean]) for st in ref.stages])
    np.testing.assert_allclose(net.run_mean.cpu().numpy(), orm, rtol=1e-4, atol=1e-5)


def _grad_rel(names, got, want):
    """Per-tensor relative error, floored at 1e-3 of the whole vector's norm."""
    total = np.sqrt(sum(float(np.sum(want[nm] ** 2)) for nm in names))
    return max(float(np.linalg.norm(got[nm] - want[nm]) / max(np.linalg.norm(want[nm]), 1e-3 * total))
               for nm in names)


def test_gradient_probes_match_oracle_and_leave_state_untouched():
    """App. B probes mid-run (fp32): PETRA and delayed tick gradients and the
    end-to-end gradient against the oracle's probes at the same state; the
    schedule then continues exactly as if no probe had run."""
    import torch
    from paper_2406_02052_amd import Net

    wl = TINY.with_(dtype="fp32")
    names, params = affine_params(wl)
    J = len(wl.widths)
    rng = np.random.default_rng(6)
    n_micro = 2 * J + 2
    imgs = [rng.standard_normal((wl.n, wl.h, wl.w, wl.c_img), dtype=np.float32) for _ in range(n_micro)]
    labs = [rng.integers(0, wl.classes, wl.n).astype(np.int32) for _ in range(n_micro)]
    ref = PetraNet([p.astype(np.float64) for p in params], names, J, wl.blocks_per_stage)
    net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype,
              input_buffer=True, param_buffer=True)
    net.set_params(params)
    net.set_optimizer(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
    net.set_backward(0)
    T = 2 * J
    for t in range(T):
        ref.tick(t, lambda m: imgs[m], lambda m: labs[m], n_micro, wl.lr, wl.momentum,
                 wl.weight_decay, wl.nesterov, wl.accum_k)
        net.tick(net.images(imgs[t]), net.labels(labs[t]))
    torch.cuda.synchronize()
    p_before = net.params.cpu().numpy().copy()
    rm_before = net.run_mean.cpu().numpy().copy()
    offs = [net.infos[i].offset for i in range(len(names))]
    def by_name(vec):
        v = vec.cpu().numpy()
        return {nm: v[o:o + int(np.prod(p.shape))].reshape(p.shape)
                for nm, o, p in zip(names, offs, params)}
    m_last = T - (J - 1)
    got = {0: by_name(net.probe_tick(0)), 3: by_name(net.probe_tick(3)),
           "e2e": by_name(net.probe_backprop(net.images(imgs[m_last]), net.labels(labs[m_last])))}
    torch.cuda.synchronize()
    want = {0: ref.probe_tick(T, lambda m: imgs[m], lambda m: labs[m], n_micro, False, False),
            3: ref.probe_tick(T, lambda m: imgs[m], lambda m: labs[m], n_micro, True, True),
            "e2e": ref.probe_backprop(imgs[m_last], labs[m_last])}
    for key in got:
        e = _grad_rel(names, got[key], want[key])
        print("probe", key, "max relative error", e, flush=True)
        assert e <= 1e-4, (key, e)
    np.testing.assert_array_equal(net.params.cpu().numpy(), p_before)
    np.testing.assert_array_equal(net.run_mean.cpu().numpy(), rm_before)
    # the schedule continues as the oracle's, which never probed
    for t in range(T, T + 2):
        ref.tick(t, lambda m: imgs[m], lambda m: labs[m], n_micro, wl.lr, wl.momentum,
                 wl.weight_decay, wl.nesterov, wl.accum_k)
        net.tick(net.images(imgs[t]), net.labels(labs[t]))
    torch.cuda.synchronize()
    want_p = {nm: p for st in ref.stages for nm, p in zip(st.names, st.params)}
    got_p = dict(zip(names, net.get_params()))
    p0 = dict(zip(names, params))
    e = _grad_rel(names, {nm: np.asarray(got_p[nm], np.float64) - p0[nm] for nm in names},
                  {nm: want_p[nm] - p0[nm] for nm in names})
    assert e <= 1e-4, e
    assert [net.stage_spans()[j][1] for j in range(J)] == [
        sum(int(np.prod(p.shape)) for nm, p in zip(names, params) if nm.startswith(f"s{j}."))
        for j in range(J)]


def test_tiny_net_fp32_accumulation_matches_oracle():
    """Gradient accumulation k = 2 in the schedule (Sec. 4.1): each stage
    updates after every second backward with the mean gradient."""
    wl = TINY.with_(dtype="fp32", accum_k=2)
    names, params = affine_params(wl)
    J = len(wl.widths)
    n_micro, ticks = 5, 5 + 2 * J
    ref, oloss, net, gloss = run_both(wl, names, params, n_micro, ticks)
    worst = compare(wl, names, params, ref, oloss, net, gloss, 1e-4, 1e-4)
    print("worst parameter increment error", worst, flush=True)


@pytest.mark.parametrize("blocks", [1, 2])
def test_split_stages_fp32_matches_oracle(blocks):
    """The per-layer split (every stem/downsampling and every block its own
    stage; J = 8 or 12): losses, parameters after every update and running
    statistics against the oracle's split schedule.  With two blocks per level
    the lower block stage rebuilds its input from the reconstruction the upper
    one sends back."""
    wl = TINY.with_(dtype="fp32", blocks_per_stage=blocks)
    names, params = affine_params(wl)
    J = len(wl.widths) * (1 + blocks)
    n_micro, ticks = 3, 3 + 2 * J
    ref, oloss, net, gloss = run_both(wl, names, params, n_micro, ticks, split=True)
    print("J", J, "losses", gloss, oloss, flush=True)
    worst = compare(wl, names, params, ref, oloss, net, gloss, 1e-4, 1e-4)
    print("worst parameter increment error", worst, flush=True)
    orm = np.concatenate([np.concatenate([m.reshape(-1) for m in st.run_mean]) for st in ref.stages])
    np.testing.assert_allclose(net.run_mean.cpu().numpy(), orm, rtol=1e-4, atol=1e-5)
    assert net.state() == (ticks, n_micro, 0)


def test_split_stages_backprop_and_delayed_variant_match_oracle():
    """Split schedule: the reversible-backprop step and the delayed-gradient
    variant (both buffers) against the oracle."""
    import torch
    from paper_2406_02052_amd import Net

    wl = TINY.with_(dtype="fp32", blocks_per_stage=2)
    names, params = affine_params(wl)
    rng = np.random.default_rng(8)
    imgs = [rng.standard_normal((wl.n, wl.h, wl.w, wl.c_img), dtype=np.float32) for _ in range(2)]
    labs = [rng.integers(0, wl.classes, wl.n).astype(np.int32) for _ in range(2)]
    ref = PetraNet([p.astype(np.float64) for p in params], names, len(wl.widths),
                   wl.blocks_per_stage, split_fronts=True)
    oloss = [ref.backprop_step(imgs[i], labs[i], wl.lr, wl.momentum, wl.weight_decay, wl.nesterov,
                               wl.accum_k) for i in range(2)]
    net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype,
              split_stages=True)
    net.set_params(params)
    net.set_optimizer(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
    gloss = []
    for i in range(2):
        net.backprop_step(net.images(imgs[i]), net.labels(labs[i]))
        torch.cuda.synchronize()
        gloss.append(float(net.loss.item()))
    compare(wl, names, params, ref, oloss, net, gloss, 1e-4, 1e-4)
    J = ref.J
    ref2, oloss2, net2, gloss2 = run_both(wl, names, params, 3, 3 + 2 * J, mode=3, split=True)
    compare(wl, names, params, ref2, oloss2, net2, gloss2, 1e-4, 1e-4)


def test_split_stages_bf16_matches_storage_oracle():
    """bf16 per-layer split (J = 12) against the storage-precision oracle:
    losses and running statistics at the stated bar, parameter increments at
    the chain bound (several reconstructed bf16 blocks deep)."""
    wl = TINY.with_(blocks_per_stage=2)
    names, params = affine_params(wl)
    J = len(wl.widths) * 3
    n_micro, ticks = 3, 3 + 2 * J
    ref, oloss, net, gloss = run_both(wl, names, params, n_micro, ticks, split=True)
    print("losses", gloss, oloss, flush=True)
    worst = compare(wl, names, params, ref, oloss, net, gloss, TOL["bf16"], CHAIN_TOL)
    print("worst parameter increment error", worst, flush=True)


# ---------------------------------------------------------------------------
# The RevNet-18-shaped schedule at its real shape (32 x 32 images, widths
# 64/128/256/512, two blocks per stage: every kernel variant the benchmark
# runs).  The batch is reduced to keep the oracle cheap; kernel selection
# depends on H, W and C only.
# ---------------------------------------------------------------------------

REAL = synth.REVNET18_SCHEDULE.with_(n=32)


def _identity_blocks(wl, params):
    """gamma = beta = 0 on the last BN of every F and G: each reversible block
    is the identity (Sec. 3.2), its reconstruction exact, and only those BNs'
    parameters get a gradient inside the blocks."""
    names = [n for n, _ in synth.net_param_shapes(wl)]
    out = list(params)
    for i, nm in enumerate(names):
        parts = nm.split(".")
        if len(parts) == 5 and parts[3] == "bn1":
            out[i] = np.zeros_like(out[i])
    return names, out


def _drained_run(wl, names, params, n_micro):
    """Feed n_micro micro-batches, then drain with petra_net_drain; the oracle
    runs the same ticks.  Returns (ref, oracle losses, net, GPU losses)."""
    import torch
    from paper_2406_02052_amd import Net

    J = len(wl.widths)
    imgs = synth.net_images(wl, n_micro)
    labs = synth.net_labels(wl, n_micro)
    bf = wl.dtype == "bf16"
    ref = PetraNet([p.astype(np.float64) for p in params], names, J, wl.blocks_per_stage,
                   weight_view=synth.round_bf16 if bf else None,
                   store=synth.round_bf16 if bf else None)
    oloss = []
    for t in range(n_micro + 2 * J - 2):
        oloss.append(ref.tick(t, lambda m: imgs[m], lambda m: labs[m], n_micro, wl.lr,
                              wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k))
    oloss = [l for l in oloss if l is not None]
    net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype)
    net.set_params(params)
    net.set_optimizer(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
    gloss = []
    for t in range(n_micro):
        if net.tick(net.images(imgs[t]), net.labels(labs[t])):
            gloss.append(float(net.loss.item()))
    tail = net.drain()
    torch.cuda.synchronize()
    gloss += [float(v) for v in tail.cpu().numpy()]
    assert net.state() == (n_micro + 2 * J - 2, n_micro, 0)
    return ref, oloss, net, gloss


def _by_name(ref, attr):
    return {nm: np.asarray(v, np.float64) for st in ref.stages
            for nm, v in zip(st.names, getattr(st, attr))}


def test_schedule_real_shape_identity_blocks_exact_gradients():
    """Drained run of 2J + 2 micro-batches with lr = 0 (every backward is exact
    backprop at the initial parameters, P8) and identity blocks: the losses,
    every tensor's momentum buffer (the momentum sum of its gradients, weight
    decay included) and the running statistics match the oracle's tick
    simulator at the stated bf16 bar; the block parameters other than the
    zeroed BNs get exactly no gradient."""
    wl = REAL.with_(lr=0.0)
    J = len(wl.widths)
    names, params = _identity_blocks(wl, synth.net_params(wl))
    ref, oloss, net, gloss = _drained_run(wl, names, params, 2 * J + 2)
    print("losses", gloss, oloss, flush=True)
    assert len(gloss) == len(oloss) == 2 * J + 2
    for a, b in zip(gloss, oloss):
        assert abs(a - b) <= TOL["bf16"] * abs(b), (a, b)
    want = _by_name(ref, "buf")
    got = dict(zip(names, net.get_momentum()))
    # Some gradients vanish in exact arithmetic.  With identity blocks the
    # gradient at the output of stage j < J-1 is the input gradient of stage
    # j+1's 1x1 stride-2 downsampling of a BN-centred gradient, whose pixel sum
    # is zero; it reaches unchanged the last BN of every block of stage j and,
    # for j > 0, stage j's own downsampling BN, so those BNs' beta gradients
    # vanish.  Stored in bf16 such a sum is rounding noise on both sides: both
    # must stay below 1e-3 of the whole momentum vector.  The other tensors are
    # compared normwise, relative to their own norm or to that 1e-3, whichever
    # is larger.
    total = np.sqrt(sum(float(np.sum(w ** 2)) for w in want.values()))
    worst = (0.0, "")
    for nm in names:
        parts = nm.split(".")
        if not np.any(want[nm] != 0):
            assert not np.any(got[nm] != 0), f"{nm}: gradient must vanish"
            continue
        j = int(parts[0][1:])
        if j < J - 1 and parts[-1] == "beta" and (
                (len(parts) == 5 and parts[3] == "bn1") or (parts[1] == "trans_bn" and j > 0)):
            assert np.linalg.norm(got[nm]) <= 1e-3 * total, (nm, np.linalg.norm(got[nm]) / total)
            assert np.linalg.norm(want[nm]) <= 1e-3 * total, nm
            continue
        e = float(np.linalg.norm(got[nm] - want[nm]) / max(np.linalg.norm(want[nm]), 1e-3 * total))
        worst = max(worst, (e, nm))
        assert e <= TOL["bf16"], (nm, e)
    print("worst momentum error", worst, flush=True)
    for nm, p0, p1 in zip(names, params, net.get_params()):
        assert np.array_equal(p0, p1), f"{nm} moved with lr = 0"
    orm = np.concatenate([np.concatenate([m.reshape(-1) for m in st.run_mean]) for st in ref.stages])
    orv = np.concatenate([np.concatenate([v.reshape(-1) for v in st.run_var]) for st in ref.stages])
    assert rel(net.run_mean.cpu().numpy(), orm) <= TOL["bf16"]
    assert rel(net.run_var.cpu().numpy(), orv) <= TOL["bf16"]


def _stage_increments(names, params, got_params, ref):
    """Per stage: (cosine, norm ratio) of the GPU's parameter increments
    against the oracle's, over the stage's whole parameter vector."""
    want = _by_name(ref, "params")
    p0 = dict(zip(names, params))
    acc = {}
    for nm, p1 in zip(names, got_params):
        s = nm.split(".")[0]
        a = (np.asarray(p1, np.float64) - p0[nm]).ravel()
        b = (want[nm] - p0[nm]).ravel()
        r = acc.setdefault(s, [0.0, 0.0, 0.0])
        r[0] += float(a @ b)
        r[1] += float(a @ a)
        r[2] += float(b @ b)
    return {s: (r[0] / np.sqrt(r[1] * r[2]), np.sqrt(r[1] / r[2])) for s, r in acc.items()}


# Fixed bounds for the trained schedule in bf16.  Training through J = 4
# stages of reconstructed bf16 blocks is chaotic: the oracle itself run in
# fp32 instead of fp64 (same storage model, batch 32) keeps the losses within
# 1 % for the first ten ticks, within 10 % to tick 20 and diverges up to 2.6x
# once the micro-batches are memorised; its per-stage increment cosine falls
# from 0.95-0.98 at tick 9 to 0.65-0.84 at tick 99 while the increment norms
# stay within 2 %.
SCHED_LOSS_EARLY = 5e-2
SCHED_COS_DRAINED = 0.8
SCHED_COS_LONG = 0.5
SCHED_NORM = 0.1


def test_schedule_real_shape_drained_run_matches_oracle():
    """The paper's setting (lr 0.1, Nesterov, weight decay 5e-4) at real shape,
    2J + 2 micro-batches fed and the pipeline drained: every loss, each stage's
    parameter increments (direction and size) and the running statistics
    against the oracle's tick simulator (measured: losses within 2.7 %, stage
    cosines 0.86-0.96, norms within 0.5 %, running mean 10 % normwise)."""
    wl = REAL
    J = len(wl.widths)
    names = [n for n, _ in synth.net_param_shapes(wl)]
    params = synth.net_params(wl)
    ref, oloss, net, gloss = _drained_run(wl, names, params, 2 * J + 2)
    print("losses", gloss, oloss, flush=True)
    assert len(gloss) == len(oloss) == 2 * J + 2
    for a, b in zip(gloss, oloss):
        assert abs(a - b) <= SCHED_LOSS_EARLY * abs(b), (a, b)
    inc = _stage_increments(names, params, net.get_params(), ref)
    print("per-stage increment cosine, norm ratio", inc, flush=True)
    for s, (c, r) in inc.items():
        assert c >= SCHED_COS_DRAINED and abs(r - 1.0) <= SCHED_NORM, (s, c, r)
    # the running statistics here follow the trained parameters (batch means
    # near zero move with the increments): chain bounds
    orm = np.concatenate([np.concatenate([m.reshape(-1) for m in st.run_mean]) for st in ref.stages])
    orv = np.concatenate([np.concatenate([v.reshape(-1) for v in st.run_var]) for st in ref.stages])
    for a, b in ((net.run_mean.cpu().numpy(), orm), (net.run_var.cpu().numpy(), orv)):
        print("running statistics", rel(a, b), cos_sim(a, b), flush=True)
        assert rel(a, b) <= CHAIN_TOL and cos_sim(a, b) >= CHAIN_COS


def test_schedule_real_shape_hundred_ticks():
    """100 ticks of the paper's setting at real shape over 8 synthetic
    micro-batches fed in turn: the losses of the first 2J + 2 micro-batches
    match the oracle; after that both runs train (the mean loss of the last 20
    ticks is below half the first losses' mean) and each stage's increment
    since the start points the oracle's way with the oracle's size."""
    import torch
    from paper_2406_02052_amd import Net

    wl = REAL
    J = len(wl.widths)
    T, D = 100, 8
    names = [n for n, _ in synth.net_param_shapes(wl)]
    params = synth.net_params(wl)
    imgs, labs = synth.net_images(wl, D), synth.net_labels(wl, D)
    ref = PetraNet([p.astype(np.float64) for p in params], names, J, wl.blocks_per_stage,
                   weight_view=synth.round_bf16, store=synth.round_bf16)
    net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype)
    net.set_params(params)
    net.set_optimizer(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
    gi = [net.images(x) for x in imgs]
    gl = [net.labels(l) for l in labs]
    oloss, gloss = [], []
    for t in range(T):
        lo = ref.tick(t, lambda m: imgs[m % D], lambda m: labs[m % D], 10 ** 9, wl.lr,
                      wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
        if net.tick(gi[t % D], gl[t % D]):
            gloss.append(float(net.loss.item()))
        if lo is not None:
            oloss.append(lo)
        if t % 20 == 0:
            print(f"tick {t}", flush=True)
    torch.cuda.synchronize()
    print("losses every 10:", [round(v, 4) for v in gloss[::10]], [round(v, 4) for v in oloss[::10]],
          flush=True)
    assert len(gloss) == len(oloss) == T - (J - 1)
    for a, b in zip(gloss[:2 * J + 2], oloss[:2 * J + 2]):
        assert abs(a - b) <= SCHED_LOSS_EARLY * abs(b), (a, b)
    first = np.mean(oloss[:2 * J + 2])
    for run in (gloss, oloss):
        assert np.isfinite(run).all()
        assert np.mean(run[-20:]) < 0.5 * first, (np.mean(run[-20:]), first)
    inc = _stage_increments(names, params, net.get_params(), ref)
    print("per-stage increment cosine, norm ratio", inc, flush=True)
    for s, (c, r) in inc.items():
        assert c >= SCHED_COS_LONG and abs(r - 1.0) <= SCHED_NORM, (s, c, r)
