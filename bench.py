"""Benchmark of PETRA's per-stage reversible step on one MI355X.

A step is one petra_stage_step call: the forward of one micro-batch and the
reconstruct + VJP of another run concurrently on two streams with the same
current parameters, then the in-place SGD update (Eq. 5).  Inputs are seeded
synthetic tensors already resident in HBM; the timed region covers exactly
--steps steps between two device synchronisations.

Prints one JSON line with the throughput (images/s per stage step), the
roofline position of the dominant kernel class (per-launch HIP events on the
launching stream, in a second pass of the same steps) and the CPU oracle's
throughput on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import synth  # noqa: E402

PEAK_HBM_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "fp32": 157.3}


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=100)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--workload", default=synth.CIFAR_STAGE.name,
                   choices=sorted(synth.STAGE_WORKLOADS) + [synth.REVNET18_SCHEDULE.name])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-profile", action="store_true")
    p.add_argument("--cpu-seconds", type=float, default=12.0,
                   help="target duration of the CPU-oracle sample")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain device copy of 256 MiB ten times (reference kernel "
                        "for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    return p.parse_args()


def copy_calibration():
    """A plain elementwise pass of known size (256 MiB read, 256 MiB written, one
    vectorized kernel per call): its FETCH_SIZE / WRITE_SIZE readings per dispatch
    calibrate the counters against bytes actually moved."""
    import torch
    n = 64 << 20
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(10):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": 4 * n, "bytes_written": 4 * n,
                      "dispatches": 10}))


def kernel_source_sha():
    """Hash of the HIP sources, to tell whether stored counter readings still
    describe the kernels that run."""
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2406_02052_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            with open(os.path.join(csrc, f), "rb") as fh:
                h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def stored_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed counter summary
    (FETCH_SIZE and WRITE_SIZE, each scaled by the copy calibration), or None
    when no reading exists or the kernel sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", "traffic_counters.md")
    if not os.path.exists(path):
        return None
    sha = kernel_source_sha()
    with open(path) as fh:
        for line in fh:
            cells = [c.strip().strip("`") for c in line.strip().strip("|").split("|")]
            if len(cells) >= 5 and cells[0] == workload and cells[1] == kernel and cells[2] == sha:
                try:
                    return float(cells[-1])
                except ValueError:
                    return None
    return None


def gpu_inputs(st, wl):
    x1, x2 = synth.stage_input(wl)
    xb1, xb2 = synth.stage_input(wl, seed_offset=10)
    g1, g2 = synth.stage_output_grad(wl)
    t = dict(xa1=st.act(x1), xa2=st.act(x2), yb1=st.act(), yb2=st.act(),
             db1=st.act(g1), db2=st.act(g2))
    # the backward micro-batch: the stage output of another micro-batch
    st.forward(st.act(xb1), st.act(xb2), t["yb1"], t["yb2"])
    for k in ("ya1", "ya2", "xr1", "xr2", "dx1", "dx2"):
        t[k] = st.act()
    return t


def one_step(st, t):
    return st.step(t["xa1"], t["xa2"], t["ya1"], t["ya2"], t["yb1"], t["yb2"], t["db1"], t["db2"],
                   t["xr1"], t["xr2"], t["dx1"], t["dx2"])


def one_step_serial(st, t):
    st.forward(t["xa1"], t["xa2"], t["ya1"], t["ya2"])
    st.reconstruct_backward(t["yb1"], t["yb2"], t["db1"], t["db2"], t["xr1"], t["xr2"],
                            t["dx1"], t["dx2"])
    st.update()


def timed(torch, fn, steps):
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return time.perf_counter() - t0


def roofline(prof, dtype):
    """Dominant kernel class (largest summed device time) against its roofline."""
    name = max(prof, key=lambda k: prof[k][1])
    n, ms, fl, by = prof[name]
    ridge = PEAK_TFLOPS[dtype] * 1e12 / (PEAK_HBM_GBS * 1e9)
    per_launch_s = ms / 1e3 / n
    if fl > 0 and fl / by >= ridge:
        achieved = fl / n / per_launch_s / 1e12
        out = {"bound": "mfma", "achieved": achieved, "peak": PEAK_TFLOPS[dtype],
               "unit": "TFLOP/s"}
    else:
        achieved = by / n / per_launch_s / 1e9
        out = {"bound": "hbm", "achieved": achieved, "peak": PEAK_HBM_GBS, "unit": "GB/s"}
    out["frac"] = out["achieved"] / out["peak"]
    out["traffic"] = None
    out["kernel"] = name
    out["launches_per_step"] = None
    out["avg_launch_us"] = per_launch_s * 1e6
    out["algorithmic_per_launch"] = {"flops": fl / n, "bytes": by / n}
    return out


def cpu_baseline(wl, target_s):
    """The oracle (fp64 numpy) timed on one stage step of a bounded sample."""
    from threadpoolctl import threadpool_info
    from oracle.stage import StageState

    names = [n for n, _ in wl.param_shapes()]
    params = synth.stage_params(wl)

    def run(n):
        w = wl.with_(n=n)
        st = StageState(params, names, 2 if wl.kind == "basic" else 3, eps=wl.bn_eps,
                        bn_momentum=wl.bn_momentum)
        x1, x2 = synth.stage_input(w)
        g1, g2 = synth.stage_output_grad(w)
        t0 = time.perf_counter()
        st.step(x1, x2, x1, x2, g1, g2, wl.lr, wl.momentum, wl.weight_decay, wl.nesterov,
                wl.accum_k)
        return time.perf_counter() - t0

    n0 = min(wl.n, 2 if wl.h * wl.w >= 3000 else 4)
    t0 = run(n0)
    n = int(min(wl.n, max(n0, n0 * target_s / max(t0, 1e-6))))
    t = run(n) if n != n0 else t0
    threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    return {"value": n / t, "unit": "images/s", "cores": threads, "kind": "oracle",
            "sample": f"one fp64 oracle stage step (forward + reconstruct/VJP + update) "
                      f"on {n} of the {wl.n} images ({t:.1f} s); BN statistics over the sample"}


def bench_schedule(args):
    """Steady-state ticks of the J-stage schedule (every stage busy every tick)."""
    import torch
    from paper_2406_02052_amd import Net

    wl = synth.REVNET18_SCHEDULE
    net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype,
              device="cuda:0")
    net.set_params(synth.net_params(wl))
    net.set_optimizer(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
    D = 8  # a synthetic dataset of 8 micro-batches, fed in turn
    imgs = [net.images(x) for x in synth.net_images(wl, D)]
    labs = [net.labels(l) for l in synth.net_labels(wl, D)]
    J = len(wl.widths)
    warm = max(args.warmup, 2 * J - 1)   # fill the pipeline first
    for t in range(warm):
        net.tick(imgs[t % D], labs[t % D])
    print(f"[bench] {wl.name}: {warm} warm-up ticks done, timing {args.steps}", file=sys.stderr,
          flush=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(warm, warm + args.steps):
        net.tick(imgs[t % D], labs[t % D])
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    loss = float(net.loss.item())
    # Reversible backpropagation on the same network and kernels (the baseline
    # of the paper's iteration-time comparison, Table 5): drain the pipeline,
    # then time as many sequential steps as ticks were timed.
    for _ in range(2 * J - 2):
        net.tick()
    for t in range(max(2, args.warmup // 4)):
        net.backprop_step(imgs[t % D], labs[t % D])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(args.steps):
        net.backprop_step(imgs[t % D], labs[t % D])
    torch.cuda.synchronize()
    el_bp = time.perf_counter() - t0
    bp_loss = float(net.loss.item())
    out = {"metric": "images/sec per stage step (fwd+reconstruct+VJP+update)",
           "value": wl.n * args.steps / el, "unit": "images/s", "n_gpus": 1,
           "steps": args.steps, "warmup": warm, "ms_per_step": el / args.steps * 1e3,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": wl.dtype,
           "data": "synthetic (seeded; CIFAR-shaped images, uniform labels over 10 classes)",
           "config": {"workload": wl.name, "batch": wl.n, "hw": [wl.h, wl.w],
                      "widths": list(wl.widths), "blocks_per_stage": wl.blocks_per_stage,
                      "stages": J, "step": "one tick: every stage's forward and backward "
                      "(delays 2(J-j)) and updates"},
           "last_loss": loss, "outputs_finite": bool(np.isfinite(loss) and np.isfinite(bp_loss)),
           "reversible_backprop": {
               "ms_per_step": el_bp / args.steps * 1e3, "value": wl.n * args.steps / el_bp,
               "unit": "images/s",
               "step": "one micro-batch: all stages' forwards, head, all stages' backwards "
                       "(blocks rebuilt from outputs) and updates, one stream",
               "iteration_time_ratio": (el_bp / args.steps) / (el / args.steps)}}
    print(json.dumps(out))


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this build runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.workload == synth.REVNET18_SCHEDULE.name:
        bench_schedule(args)
        return
    import torch
    from paper_2406_02052_amd import Stage, petra_stage_profile, petra_stage_profile_read

    wl = synth.STAGE_WORKLOADS[args.workload]
    st = Stage(wl.n, wl.h, wl.w, wl.c_half, wl.blocks, wl.kind, wl.dtype, c_mid=wl.c_mid,
               bn_eps=wl.bn_eps, bn_momentum=wl.bn_momentum, device="cuda:0")
    st.set_params(synth.stage_params(wl))
    st.set_optimizer(lr=wl.lr, momentum=wl.momentum, weight_decay=wl.weight_decay,
                     nesterov=wl.nesterov, accum_k=wl.accum_k)
    t = gpu_inputs(st, wl)
    for _ in range(args.warmup):
        one_step(st, t)
    print(f"[bench] {wl.name}: warm-up done, timing {args.steps} steps", file=sys.stderr,
          flush=True)
    el = timed(torch, lambda: one_step(st, t), args.steps)
    el_serial = timed(torch, lambda: one_step_serial(st, t), args.steps)
    ms = el / args.steps * 1e3
    out = {"metric": "images/sec per stage step (fwd+reconstruct+VJP+update)",
           "value": wl.n * args.steps / el, "unit": "images/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": ms,
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": wl.dtype, "data": "synthetic (seeded; CIFAR/ImageNet-shaped tensors)",
           "config": {"workload": wl.name, "batch": wl.n, "hw": [wl.h, wl.w],
                      "channels": 2 * wl.c_half, "blocks": wl.blocks, "block": wl.kind,
                      "mid_channels": wl.c_mid or None,
                      "step": "forward || reconstruct+VJP on two streams, then SGD update"},
           "serial_ms_per_step": el_serial / args.steps * 1e3}
    if not args.no_profile:
        petra_stage_profile(st.handle, True)
        for _ in range(args.steps):
            one_step(st, t)
        torch.cuda.synchronize()
        prof = {k: v for k, v in petra_stage_profile_read(st.handle).items() if v[0] > 0}
        petra_stage_profile(st.handle, False)
        rl = roofline(prof, wl.dtype)
        rl["launches_per_step"] = prof[rl["kernel"]][0] / args.steps
        rl["traffic"] = stored_traffic(wl.name, rl["kernel"])
        rl["kernel_source_sha"] = kernel_source_sha()
        out["roofline"] = rl
        out["kernels"] = {k: {"launches_per_step": v[0] / args.steps,
                              "avg_us": v[1] * 1e3 / v[0],
                              "tflops": v[2] / (v[1] / 1e3) / 1e12 if v[2] else 0.0,
                              "gbs": v[3] / (v[1] / 1e3) / 1e9,
                              "share": v[1] / sum(p[1] for p in prof.values())}
                          for k, v in sorted(prof.items(), key=lambda kv: -kv[1][1])}
        conv_ms = sum(prof[k][1] for k in prof if k.startswith("conv_"))
        conv_fl = sum(prof[k][2] for k in prof if k.startswith("conv_"))
        out["mfma_util_pct"] = 100.0 * conv_fl / (conv_ms / 1e3) / (PEAK_TFLOPS[wl.dtype] * 1e12)
    finite = all(bool(torch.isfinite(t[k].float()).all()) for k in ("ya1", "xr1", "dx2"))
    out["outputs_finite"] = finite
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
