"""Benchmark of PETRA's per-stage reversible step on one MI355X.

A step is one petra_stage_step call: the forward of one micro-batch and the
reconstruct + VJP of another run concurrently on two streams with the same
current parameters, then the in-place SGD update (Eq. 5).  Inputs are seeded
synthetic tensors already resident in HBM; the timed region covers exactly
--steps steps between two device synchronisations.

The headline is the ImageNet-shaped RevNet-50 bottleneck stage (64 x 56 x 56,
256 channels, 3 blocks); the CIFAR- and ImageNet32-shaped stages and the
four-stage schedule follow in the same run under "configs", each with its own
figures.  Per stage workload: throughput, the serialized step, a cold-cache
variant, the roofline position of the dominant kernel (per-launch HIP events
on the launching stream, in a second pass of the same steps), the
convolutions' MFMA fraction and the BN / elementwise kernels' HBM fraction,
and the CPU oracle's throughput on a bounded sample (fp64 and fp32).  Prints
one JSON line.
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
    p.add_argument("--workload", default=synth.IMAGENET_BOTTLENECK_STAGE.name,
                   choices=sorted(synth.STAGE_WORKLOADS) + [synth.REVNET18_SCHEDULE.name],
                   help="the headline workload (default: the ImageNet-shaped bottleneck stage)")
    p.add_argument("--only", action="store_true",
                   help="time the headline workload alone (no nested lines for the others)")
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-profile", action="store_true")
    p.add_argument("--no-cold", action="store_true", help="skip the cold-cache variant")
    p.add_argument("--cpu-seconds", type=float, default=6.0,
                   help="target duration of each CPU-oracle sample")
    p.add_argument("--gradient-quality", action="store_true",
                   help="train the schedule (PETRA backward, both buffers kept) and report "
                        "per-stage cosine similarity / norm ratio of the PETRA, delayed and "
                        "end-to-end gradients at snapshots (App. B)")
    p.add_argument("--gq-ticks", type=int, default=240)
    p.add_argument("--gq-every", type=int, default=20)
    p.add_argument("--memory-report", action="store_true",
                   help="per-stage device bytes of the schedule with the buffers on/off and "
                        "the 18-stage RevNet-50 estimate (Tables 3 and 6); host only")
    p.add_argument("--k-sweep", default=None,
                   help="comma-separated accumulation factors: schedule throughput and loss "
                        "per k with lr = 0.1 * batch * k / 256")
    p.add_argument("--copy-calibration", action="store_true",
                   help="only run a plain device copy of 256 MiB ten times (reference kernel "
                        "for scaling the FETCH_SIZE / WRITE_SIZE counters)")
    p.add_argument("--counters-summary", nargs=5, metavar=("WORKLOAD", "FETCH_DIR", "WRITE_DIR",
                                                           "COPY_FETCH_DIR", "COPY_WRITE_DIR"),
                   help="host only: from rocprofv3 --pmc FETCH_SIZE / WRITE_SIZE csv output of "
                        "the bench command and of --copy-calibration, write the calibrated HBM "
                        "bytes per dispatch of every kernel into profiles/traffic.json")
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


TRAFFIC_JSON = os.path.join(ROOT, "profiles", "traffic.json")


def short_kernel_name(name: str) -> str:
    """'void petra::k<1, 2>(petra::Args)' -> 'petra::k<1, 2>' (the profiler's
    form): the argument list is the last parenthesised group outside template
    brackets."""
    if name.startswith("void "):
        name = name[5:]
    depth, cut = 0, -1
    for i, ch in enumerate(name):
        depth += ch == "<"
        depth -= ch == ">"
        if ch == "(" and depth == 0:
            cut = i
    return name if cut < 0 else name[:cut]


def _pmc_rows(d, counter):
    """{kernel: [values per dispatch]} from a rocprofv3 --pmc csv directory."""
    import csv
    import glob
    out = {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] == counter:
                    out.setdefault(short_kernel_name(r["Kernel_Name"]), []).append(
                        float(r["Counter_Value"]))
    return out


def counters_summary(workload, fetch_dir, write_dir, copy_fetch_dir, copy_write_dir):
    """Calibrated HBM bytes per dispatch of every kernel of a workload's bench
    run, stored in profiles/traffic.json under the current kernel-source hash."""
    fetch, write = _pmc_rows(fetch_dir, "FETCH_SIZE"), _pmc_rows(write_dir, "WRITE_SIZE")
    copy_bytes = 256 << 20
    cf = [v for k, vs in _pmc_rows(copy_fetch_dir, "FETCH_SIZE").items() if "neg" in k.lower()
          for v in vs]
    cw = [v for k, vs in _pmc_rows(copy_write_dir, "WRITE_SIZE").items() if "neg" in k.lower()
          for v in vs]
    ff = copy_bytes / (1024.0 * float(np.median(cf)))
    fw = copy_bytes / (1024.0 * float(np.median(cw)))
    sha = kernel_source_sha()
    data = {"entries": []}
    if os.path.exists(TRAFFIC_JSON):
        with open(TRAFFIC_JSON) as fh:
            data = json.load(fh)
    data["entries"] = [e for e in data["entries"] if e["workload"] != workload]
    for k in sorted(set(fetch) & set(write)):
        if not k.startswith("petra::"):
            continue
        f_kib, w_kib = float(np.mean(fetch[k])), float(np.mean(write[k]))
        data["entries"].append({
            "workload": workload, "kernel": k, "kernel_source_sha": sha,
            "dispatches": len(fetch[k]), "fetch_kib": f_kib, "write_kib": w_kib,
            "fetch_factor": ff, "write_factor": fw,
            "hbm_bytes_per_launch": 1024.0 * (f_kib * ff + w_kib * fw)})
    data["calibration"] = ("one torch.neg dispatch over 256 MiB (reads and writes 256 MiB); "
                           "factor = bytes moved / (counter KiB x 1024)")
    with open(TRAFFIC_JSON, "w") as fh:
        json.dump(data, fh, indent=1)
        fh.write("\n")
    print(json.dumps({"workload": workload, "kernel_source_sha": sha, "fetch_factor": ff,
                      "write_factor": fw, "kernels": len(data["entries"])}))


def stored_traffic(workload, kernel):
    """Calibrated HBM bytes per launch of `kernel` from profiles/traffic.json,
    or None when no reading exists or the kernel sources changed since."""
    if not os.path.exists(TRAFFIC_JSON):
        return None
    with open(TRAFFIC_JSON) as fh:
        data = json.load(fh)
    sha = kernel_source_sha()
    for e in data.get("entries", []):
        if e["workload"] == workload and e["kernel"] == kernel and e["kernel_source_sha"] == sha:
            return e["hbm_bytes_per_launch"]
    return None


def gpu_inputs(st, wl):
    x1, x2 = synth.stage_input(wl)
    xb1, xb2 = synth.stage_input(wl, seed_offset=10)
    g1, g2 = synth.stage_output_grad(wl)
    t = dict(xa1=st.act(x1), xa2=st.act(x2), yb1=st.act(), yb2=st.act(),
             db1=st.act(g1), db2=st.act(g2), nb1=st.act(-g1), nb2=st.act(-g2), flip=0)
    # the backward micro-batch: the stage output of another micro-batch
    st.forward(st.act(xb1), st.act(xb2), t["yb1"], t["yb2"])
    for k in ("ya1", "ya2", "xr1", "xr2", "dx1", "dx2"):
        t[k] = st.act()
    return t


def output_grad(t):
    """The backward micro-batch's output gradient for the next step.

    Its sign alternates from step to step.  A fixed synthetic gradient is not
    the gradient of any loss: applied every step at the workload's learning
    rate it pushes the weights the same way without end, and the activations
    grow geometrically (non-finite after about a hundred steps).  With the sign
    alternating, momentum SGD oscillates about the initial weights; every step
    does the same work."""
    t["flip"] ^= 1
    return (t["db1"], t["db2"]) if t["flip"] else (t["nb1"], t["nb2"])


def one_step(st, t):
    d1, d2 = output_grad(t)
    return st.step(t["xa1"], t["xa2"], t["ya1"], t["ya2"], t["yb1"], t["yb2"], d1, d2,
                   t["xr1"], t["xr2"], t["dx1"], t["dx2"])


def one_step_serial(st, t):
    d1, d2 = output_grad(t)
    st.forward(t["xa1"], t["xa2"], t["ya1"], t["ya2"])
    st.reconstruct_backward(t["yb1"], t["yb2"], d1, d2, t["xr1"], t["xr2"], t["dx1"], t["dx2"])
    st.update()


def timed(torch, fn, steps):
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    return time.perf_counter() - t0


def cold_cache_ms(torch, st, t, steps):
    """Mean step time with the caches cold: before every step a 512 MiB buffer
    (twice the 256 MB last-level cache) is rewritten, and only the step itself
    is timed (HIP events on the stream the step is ordered on)."""
    flush = torch.empty(128 << 20, dtype=torch.float32, device="cuda:0")
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    torch.cuda.synchronize()
    for a, b in evs:
        flush.fill_(1.0)
        a.record()
        one_step(st, t)
        b.record()
    torch.cuda.synchronize()
    return float(np.mean([a.elapsed_time(b) for a, b in evs])), flush.numel() * 4


# Kernel classes bound by launch latency, not by HBM or MFMA: the BN finalizes
# (one small block per channel reducing the partial rows, ~0.15-2 MB per
# launch in ~4-5 us).  They take no part in the choice of the roofline kernel;
# when one of them has the largest summed time it is reported beside it.
LAUNCH_BOUND_CLASSES = (4, 5)   # K_BN_FINALIZE, K_BN_BWD_FINALIZE


def roofline(kernels, dtype):
    """Dominant kernel (largest summed device time among the kernels an HBM or
    MFMA roofline bounds) against its roofline."""
    bounded = [k for k in kernels if k[1] not in LAUNCH_BOUND_CLASSES] or list(kernels)
    name, cls, n, ms, fl, by = max(bounded, key=lambda k: k[3])
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
    out["kernel_class"] = cls
    out["launches"] = n
    out["avg_launch_us"] = per_launch_s * 1e6
    out["algorithmic_per_launch"] = {"flops": fl / n, "bytes": by / n}
    return out


CONV_CLASSES = ("conv_fprop", "conv_dgrad", "conv_wgrad")
HBM_CLASSES = ("bn_finalize", "bn_bwd_finalize", "combine_fwd", "combine_bwd")


def targets(prof, dtype):
    """The convolutions' MFMA fraction and the BN / elementwise kernels' HBM
    fraction, each over all their launches (summed algorithmic flops or bytes
    over summed device time), against the peak and the stated targets."""
    def frac(classes, idx, peak):
        t = sum(prof[k][1] for k in classes if k in prof) / 1e3
        q = sum(prof[k][idx] for k in classes if k in prof)
        return (q / t / peak) if t > 0 else None
    return {"conv_mfma_frac": frac(CONV_CLASSES, 2, PEAK_TFLOPS[dtype] * 1e12),
            "conv_mfma_target": 0.5,
            "bn_elementwise_hbm_frac": frac(HBM_CLASSES, 3, PEAK_HBM_GBS * 1e9),
            "bn_elementwise_hbm_target": 0.7}


def _threads():
    from threadpoolctl import threadpool_info
    return max([i.get("num_threads", 1) for i in threadpool_info()] or [1])


def cpu_baseline(wl, target_s):
    """The oracle timed on one stage step of a bounded sample: fp64 (the
    parity oracle) and fp32."""
    from oracle.stage import StageState

    names = [n for n, _ in wl.param_shapes()]
    params = synth.stage_params(wl)

    def run(n, dtype):
        w = wl.with_(n=n)
        st = StageState(params, names, 2 if wl.kind == "basic" else 3, eps=wl.bn_eps,
                        bn_momentum=wl.bn_momentum, dtype=dtype)
        x1, x2 = synth.stage_input(w)
        g1, g2 = synth.stage_output_grad(w)
        t0 = time.perf_counter()
        st.step(x1, x2, x1, x2, g1, g2, wl.lr, wl.momentum, wl.weight_decay, wl.nesterov,
                wl.accum_k)
        return time.perf_counter() - t0

    res = {}
    for dtype, key in ((np.float64, "fp64"), (np.float32, "fp32")):
        n0 = min(wl.n, 2 if wl.h * wl.w >= 3000 else 4)
        t0 = run(n0, dtype)
        n = int(min(wl.n, max(n0, n0 * target_s / max(t0, 1e-6))))
        t = run(n, dtype) if n != n0 else t0
        res[key] = (n, t)
    (n, t), (n32, t32) = res["fp64"], res["fp32"]
    return {"value": n / t, "unit": "images/s", "cores": _threads(), "kind": "oracle",
            "sample": f"one fp64 oracle stage step (forward + reconstruct/VJP + update) on {n} "
                      f"of the {wl.n} images ({t:.1f} s); BN statistics over the sample",
            "fp32": {"value": n32 / t32, "unit": "images/s",
                     "sample": f"the same step in fp32 on {n32} images ({t32:.1f} s)"}}


def bench_stage(args, wl, cpu=True, cold=True):
    """One stage workload: petra_stage_step throughput, serialized step, the
    per-kernel profile with the roofline of the dominant kernel, the cold-cache
    variant and the CPU oracle."""
    import torch
    from paper_2406_02052_amd import (Stage, petra_stage_profile, petra_stage_profile_kernel,
                                      petra_stage_profile_read)

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
    if cold:
        cms, fb = cold_cache_ms(torch, st, t, max(10, args.steps // 4))
        out["cold_cache"] = {"ms_per_step": cms, "value": wl.n / (cms / 1e3), "unit": "images/s",
                             "flush_bytes_before_each_step": fb,
                             "note": "each step timed alone after rewriting a buffer twice "
                                     "the size of the last-level cache"}
    if not args.no_profile:
        # per-launch durations from a pass of the same steps with every launch
        # on one stream (forward, backward, update in order), so each timed
        # launch has the device to itself as in a kernel trace
        petra_stage_profile(st.handle, True)
        for _ in range(args.steps):
            one_step_serial(st, t)
        torch.cuda.synchronize()
        prof = {k: v for k, v in petra_stage_profile_read(st.handle).items() if v[0] > 0}
        kern = petra_stage_profile_kernel(st.handle)
        petra_stage_profile(st.handle, False)
        rl = roofline(kern, wl.dtype)
        rl["launches_per_step"] = rl.pop("launches") / args.steps
        rl["traffic"] = stored_traffic(wl.name, rl["kernel"])
        rl["kernel_source_sha"] = kernel_source_sha()
        top = max(kern, key=lambda k: k[3])
        if top[0] != rl["kernel"]:
            # the largest summed time belongs to a launch-bound kernel
            rl["dominant_by_time"] = {
                "kernel": top[0], "kernel_class": top[1], "bound": "launch",
                "launches_per_step": top[2] / args.steps, "avg_launch_us": top[3] * 1e3 / top[2],
                "share": top[3] / sum(k[3] for k in kern)}
        out["roofline"] = rl
        out["kernels"] = {name: {"class": cls, "launches_per_step": n / args.steps,
                                 "avg_us": m * 1e3 / n,
                                 "tflops": f / (m / 1e3) / 1e12 if f else 0.0,
                                 "gbs": b / (m / 1e3) / 1e9,
                                 "share": m / sum(k[3] for k in kern)}
                          for name, cls, n, m, f, b in sorted(kern, key=lambda k: -k[3])}
        out["kernel_classes"] = {k: {"launches_per_step": v[0] / args.steps,
                                     "avg_us": v[1] * 1e3 / v[0], "share":
                                     v[1] / sum(p[1] for p in prof.values())}
                                 for k, v in sorted(prof.items(), key=lambda kv: -kv[1][1])}
        out["targets"] = targets(prof, wl.dtype)
        conv_ms = sum(prof[k][1] for k in prof if k in CONV_CLASSES)
        conv_fl = sum(prof[k][2] for k in prof if k in CONV_CLASSES)
        out["mfma_util_pct"] = 100.0 * conv_fl / (conv_ms / 1e3) / (PEAK_TFLOPS[wl.dtype] * 1e12)
    finite = all(bool(torch.isfinite(t[k].float()).all()) for k in ("ya1", "xr1", "dx2"))
    out["outputs_finite"] = finite
    if cpu:
        out["cpu_baseline"] = cpu_baseline(wl, args.cpu_seconds)
    del st
    return out


def cpu_baseline_schedule(target_s):
    """The oracle's tick simulator timed over 2J+2 ticks of the schedule on a
    bounded batch (fp64 and fp32), per tick."""
    from oracle.net import PetraNet

    wl = synth.REVNET18_SCHEDULE
    names = [nm for nm, _ in synth.net_param_shapes(wl)]
    params = [p.astype(np.float64) for p in synth.net_params(wl)]
    J = len(wl.widths)

    def run(n, dtype, ticks):
        w = wl.with_(n=n)
        imgs = synth.net_images(w, ticks)
        labs = synth.net_labels(w, ticks)
        ref = PetraNet(params, names, J, wl.blocks_per_stage, dtype=dtype)
        t0 = time.perf_counter()
        for t in range(ticks):
            ref.tick(t, lambda m: imgs[m], lambda m: labs[m], ticks, wl.lr, wl.momentum,
                     wl.weight_decay, wl.nesterov, wl.accum_k)
        return (time.perf_counter() - t0) / ticks

    res = {}
    for dtype, key in ((np.float64, "fp64"), (np.float32, "fp32")):
        per = run(2, dtype, 2)
        n = int(min(wl.n, max(2, 2 * target_s / max(per * (2 * J + 2), 1e-6))))
        res[key] = (n, run(n, dtype, 2 * J + 2))
    (n, t), (n32, t32) = res["fp64"], res["fp32"]
    return {"value": n / t, "unit": "images/s", "cores": _threads(), "kind": "oracle",
            "sample": f"fp64 tick simulator, {2 * J + 2} ticks (pipeline fill and steady "
                      f"state) on {n} of the {wl.n} images, {t:.2f} s per tick",
            "fp32": {"value": n32 / t32, "unit": "images/s",
                     "sample": f"the same in fp32 on {n32} images, {t32:.2f} s per tick"}}


def bench_schedule(args, cpu=True):
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
    del net
    # The paper's per-layer split of the same network (every stem/downsampling
    # and every block its own stage): more, smaller stages in the pipeline.
    snet = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype,
               device="cuda:0", split_stages=True)
    snet.set_params(synth.net_params(wl))
    snet.set_optimizer(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, wl.accum_k)
    SJ = snet.n_stages
    swarm = max(args.warmup, 2 * SJ - 1)
    for t in range(swarm):
        snet.tick(imgs[t % D], labs[t % D])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(swarm, swarm + args.steps):
        snet.tick(imgs[t % D], labs[t % D])
    torch.cuda.synchronize()
    el_split = time.perf_counter() - t0
    split_loss = float(snet.loss.item())
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
               "iteration_time_ratio": (el_bp / args.steps) / (el / args.steps)},
           "split_stages": {
               "stages": SJ, "ms_per_tick": el_split / args.steps * 1e3,
               "value": wl.n * args.steps / el_split, "unit": "images/s",
               "last_loss": split_loss,
               "step": "one tick of the per-layer split (stem, downsamplings and blocks as "
                       "stages, delays 2(J-1-j))"}}
    out["outputs_finite"] = out["outputs_finite"] and bool(np.isfinite(split_loss))
    del snet
    if cpu:
        out["cpu_baseline"] = cpu_baseline_schedule(args.cpu_seconds)
    return out


def _cos(a, b):
    na, nb = float(np.linalg.norm(a)), float(np.linalg.norm(b))
    return float(np.dot(a.astype(np.float64), b.astype(np.float64)) / (na * nb)) if na and nb else 0.0


def gradient_quality(args):
    """App. B analog on synthetic data: the schedule trains with the PETRA
    backward while keeping both buffers; every gq_every ticks the gradients the
    next tick would produce as PETRA and as the standard delayed gradient, and
    the end-to-end gradient of each stage's micro-batch at the current
    parameters, are probed and compared per stage (cosine similarity, norm
    ratio).  Host-side numpy on the probed vectors."""
    import torch
    from paper_2406_02052_amd import BWD_DELAYED, BWD_RECONSTRUCT, Net

    wl = synth.REVNET18_SCHEDULE
    net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes, wl.dtype,
              device="cuda:0", input_buffer=True, param_buffer=True)
    net.set_params(synth.net_params(wl))
    net.set_optimizer(wl.lr, wl.momentum, wl.weight_decay, wl.nesterov, 1)
    net.set_backward(BWD_RECONSTRUCT)
    D = 32
    imgs = [net.images(x) for x in synth.net_images(wl, D)]
    labs = [net.labels(l) for l in synth.net_labels(wl, D)]
    J = len(wl.widths)
    spans = net.stage_spans()
    keys = ["cos_petra_delayed", "cos_petra_e2e", "cos_delayed_e2e", "norm_petra_delayed",
            "norm_petra_e2e", "norm_delayed_e2e"]
    snaps = []
    for t in range(args.gq_ticks):
        if t >= 2 * J and t % args.gq_every == 0:
            gp = net.probe_tick(BWD_RECONSTRUCT).cpu().numpy()
            gd = net.probe_tick(BWD_DELAYED).cpu().numpy()
            rows = []
            for j, (o, n) in enumerate(spans):
                mb = t - (2 * J - 2 - j)
                ge = net.probe_backprop(imgs[mb % D], labs[mb % D]).cpu().numpy()[o:o + n]
                a, b = gp[o:o + n], gd[o:o + n]
                na, nb, ne = (float(np.linalg.norm(v)) for v in (a, b, ge))
                rows.append(dict(zip(keys, [_cos(a, b), _cos(a, ge), _cos(b, ge),
                                            na / nb if nb else 0.0, na / ne if ne else 0.0,
                                            nb / ne if ne else 0.0])))
            torch.cuda.synchronize()
            snaps.append({"tick": t, "loss": float(net.loss.item()), "stages": rows})
            print(f"[gq] tick {t} loss {snaps[-1]['loss']:.4f} cos(petra,delayed) "
                  + " ".join(f"{r['cos_petra_delayed']:.4f}" for r in rows), file=sys.stderr,
                  flush=True)
        net.tick(imgs[t % D], labs[t % D])
    torch.cuda.synchronize()
    mean = [{k: float(np.mean([s["stages"][j][k] for s in snaps])) for k in keys} for j in range(J)]
    out = {"metric": "gradient approximation quality per stage (App. B)",
           "config": {"workload": wl.name, "batch": wl.n, "widths": list(wl.widths),
                      "blocks_per_stage": wl.blocks_per_stage, "stages": J, "lr": wl.lr,
                      "accum_k": 1, "ticks": args.gq_ticks, "every": args.gq_every,
                      "data": "32 synthetic micro-batches (N(0,1) images, uniform labels) in turn",
                      "dtype": wl.dtype},
           "delay_per_stage": [2 * (J - 1 - j) for j in range(J)],
           "mean_over_snapshots": mean, "snapshots": snaps}
    print(json.dumps(out))


def memory_report():
    """Tables 3 and 6 analogs: the library's plan per stage (bytes by purpose)
    for the RevNet-18 schedule with the input/parameter buffers on and off, and
    the host-side estimate for an 18-stage RevNet-50 on ImageNet at batch 64."""
    from paper_2406_02052_amd import _lib as L
    from paper_2406_02052_amd import memory as M
    from paper_2406_02052_amd.stage import ctypes_int_array

    wl = synth.REVNET18_SCHEDULE
    lib = {}
    for ib, pb in ((True, True), (True, False), (False, True), (False, False)):
        desc = L.NetDesc(wl.n, wl.h, wl.w, wl.c_img, len(wl.widths), ctypes_int_array(wl.widths),
                         wl.blocks_per_stage, wl.classes, L.PETRA_BF16, wl.bn_eps, wl.bn_momentum,
                         int(ib), int(pb))
        h = L.petra_net_create(desc)
        rows = [L.petra_net_memory(h, j) for j in range(len(wl.widths))]
        L.petra_net_destroy(h)
        lib[f"input_buffer={int(ib)},param_buffer={int(pb)}"] = {
            "per_stage": rows, "total": sum(r["total"] for r in rows)}
    base = lib["input_buffer=1,param_buffer=1"]["total"]
    for v in lib.values():
        v["saving_pct"] = 100.0 * (1.0 - v["total"] / base)
    est = M.revnet50_imagenet_18(64)
    out = {"metric": "device bytes per stage by purpose (Tables 3 and 6)",
           "schedule": {"workload": wl.name, "dtype": wl.dtype, "settings": lib},
           "revnet50_imagenet_18_stages_batch64_estimate": {
               "act_bytes": 4, "per_stage_petra": M.estimate(est, False, False),
               "savings": M.savings_table(est)}}
    print(json.dumps(out))


def k_sweep(args):
    """Accumulation sweep (Sec. 4.1, Fig. 3 mechanism): per k, the schedule's
    tick time and the loss over a fixed number of micro-batches of synthetic
    data, with the learning rate scaled linearly with the effective batch and
    warmed up linearly over the first quarter of the ticks."""
    import torch
    from paper_2406_02052_amd import Net

    wl = synth.REVNET18_SCHEDULE
    D = 8
    J = len(wl.widths)
    res = []
    for k in [int(v) for v in args.k_sweep.split(",")]:
        net = Net(wl.n, wl.h, wl.w, wl.c_img, wl.widths, wl.blocks_per_stage, wl.classes,
                  wl.dtype, device="cuda:0")
        net.set_params(synth.net_params(wl))
        lr = 0.1 * wl.n * k / 256
        warm = max(1, args.steps // 4)   # linear warm-up of the scaled rate (large-batch recipe)
        imgs = [net.images(x) for x in synth.net_images(wl, D)]
        labs = [net.labels(l) for l in synth.net_labels(wl, D)]
        losses = []
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for t in range(args.steps):
            if t <= warm:
                net.set_optimizer(lr * min(1.0, (t + 1) / warm), wl.momentum, wl.weight_decay,
                                  wl.nesterov, k)
            if net.tick(imgs[t % D], labs[t % D]) and (t % 8 == 0 or t == args.steps - 1):
                losses.append(float(net.loss.item()))
        torch.cuda.synchronize()
        el = time.perf_counter() - t0
        res.append({"k": k, "lr": lr, "warmup_ticks": warm, "ms_per_tick": el / args.steps * 1e3,
                    "images_per_s": wl.n * args.steps / el, "loss_first": losses[0],
                    "loss_last": losses[-1], "finite": bool(np.isfinite(losses[-1]))})
        print(f"[k-sweep] k={k} {res[-1]['ms_per_tick']:.3f} ms/tick loss {losses[0]:.3f} -> "
              f"{losses[-1]:.3f}", file=sys.stderr, flush=True)
        del net
    print(json.dumps({"metric": "accumulation sweep of the schedule", "workload": wl.name,
                      "ticks": args.steps, "stages": J,
                      "data": "8 synthetic micro-batches in turn", "results": res}))


def main():
    args = parse()
    if args.counters_summary:
        counters_summary(*args.counters_summary)
        return
    if args.copy_calibration:
        copy_calibration()
        return
    if args.gpus != 1:
        print(json.dumps({"error": "bench.py runs on one GPU only; --gpus must be 1",
                          "n_gpus": args.gpus}))
        sys.exit(2)
    if args.memory_report:
        memory_report()
        return
    if args.gradient_quality:
        gradient_quality(args)
        return
    if args.k_sweep:
        k_sweep(args)
        return
    cpu = not args.no_cpu_baseline
    sched = synth.REVNET18_SCHEDULE.name
    if args.workload == sched:
        out = bench_schedule(args, cpu=cpu)
    else:
        out = bench_stage(args, synth.STAGE_WORKLOADS[args.workload], cpu=cpu,
                          cold=not args.no_cold)
    if not args.only:
        # the other workloads of the build, each with its own line of figures
        out["configs"] = {}
        for name in (synth.CIFAR_STAGE.name, synth.IMAGENET32_STAGE.name,
                     synth.IMAGENET_BOTTLENECK_STAGE.name, sched):
            if name == args.workload:
                continue
            if name == sched:
                out["configs"][name] = bench_schedule(args, cpu=cpu)
            else:
                out["configs"][name] = bench_stage(args, synth.STAGE_WORKLOADS[name], cpu=cpu,
                                                   cold=not args.no_cold)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
