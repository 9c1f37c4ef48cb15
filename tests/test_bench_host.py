"""Host-side logic of bench.py (no GPU)."""
import numpy as np

import bench


def test_stage_bench_output_gradient_alternates_sign():
    """The stage bench feeds a fixed synthetic output gradient; applied every
    step with the same sign, momentum SGD drives the weights without bound, so
    consecutive steps must see g and -g in turn."""
    g1 = np.arange(6, dtype=np.float32).reshape(2, 3)
    g2 = -2.0 * g1
    t = dict(db1=g1, db2=g2, nb1=-g1, nb2=-g2, flip=0)
    seen = [bench.output_grad(t) for _ in range(4)]
    assert seen[0][0] is g1 and seen[0][1] is g2
    assert seen[2][0] is g1 and seen[2][1] is g2
    for d1, d2 in (seen[1], seen[3]):
        assert np.array_equal(d1, -g1) and np.array_equal(d2, -g2)
    # over a pair of steps the gradients cancel exactly
    assert np.array_equal(seen[0][0] + seen[1][0], np.zeros_like(g1))



def test_short_kernel_name_matches_the_profilers_form():
    assert (bench.short_kernel_name("void petra::conv_halo_kernel<8, 32, 32, 4, 1, 0, 1, true>"
                                    "(petra::ConvArgs)")
            == "petra::conv_halo_kernel<8, 32, 32, 4, 1, 0, 1, true>")
    assert bench.short_kernel_name("petra::sgd_kernel(float*, int)") == "petra::sgd_kernel"
    # parentheses inside template arguments or a namespace name are kept
    assert bench.short_kernel_name("void k<(int)3>(int)") == "k<(int)3>"
    assert (bench.short_kernel_name("void petra::(anonymous namespace)::k<4>(float*)")
            == "petra::(anonymous namespace)::k<4>")


def _pmc_csv(path, rows):
    import csv
    import os
    os.makedirs(path, exist_ok=True)
    with open(os.path.join(path, "run_counter_collection.csv"), "w", newline="") as fh:
        w = csv.writer(fh)
        w.writerow(["Kernel_Name", "Counter_Name", "Counter_Value"])
        for r in rows:
            w.writerow(r)


def test_counters_summary_calibrates_and_stored_traffic_reads_it(tmp_path, monkeypatch):
    """The counter summary scales FETCH_SIZE / WRITE_SIZE per dispatch by the
    plain copy's readings and is read back only under the same source hash."""
    monkeypatch.setattr(bench, "TRAFFIC_JSON", str(tmp_path / "traffic.json"))
    k = "void petra::conv1x1_kernel<128, 32, 0>(petra::ConvArgs, int)"
    _pmc_csv(tmp_path / "f", [(k, "FETCH_SIZE", 1000.0), (k, "FETCH_SIZE", 3000.0),
                              ("void at::native::other()", "FETCH_SIZE", 5.0)])
    _pmc_csv(tmp_path / "w", [(k, "WRITE_SIZE", 500.0), (k, "WRITE_SIZE", 500.0)])
    # the copy reads and writes 256 MiB; FETCH_SIZE reads half of it, WRITE_SIZE all
    neg = "void at::native::vectorized_elementwise_kernel<4, neg>(int)"
    _pmc_csv(tmp_path / "cf", [(neg, "FETCH_SIZE", 131072.0)] * 3)
    _pmc_csv(tmp_path / "cw", [(neg, "WRITE_SIZE", 262144.0)] * 3)
    bench.counters_summary("wl", str(tmp_path / "f"), str(tmp_path / "w"), str(tmp_path / "cf"),
                           str(tmp_path / "cw"))
    got = bench.stored_traffic("wl", "petra::conv1x1_kernel<128, 32, 0>")
    assert got == 1024.0 * (2000.0 * 2.0 + 500.0 * 1.0)
    assert bench.stored_traffic("other", "petra::conv1x1_kernel<128, 32, 0>") is None
    monkeypatch.setattr(bench, "kernel_source_sha", lambda: "0000000000000000")
    assert bench.stored_traffic("wl", "petra::conv1x1_kernel<128, 32, 0>") is None


def test_roofline_picks_the_kernel_with_most_device_time():
    kernels = [("a", 0, 10, 1.0, 1e9, 1e9), ("b", 6, 4, 2.0, 0.0, 4.0e8)]
    rl = bench.roofline(kernels, "bf16")
    assert rl["kernel"] == "b" and rl["bound"] == "hbm"
    # 1e8 bytes per launch in 0.5 ms -> 200 GB/s
    assert abs(rl["achieved"] - 200.0) < 1e-9 and abs(rl["frac"] - 200.0 / 8000.0) < 1e-12
    rl = bench.roofline([("c", 0, 1, 1.0, 1e12, 1e9)], "bf16")
    assert rl["bound"] == "mfma" and abs(rl["achieved"] - 1000.0) < 1e-9


def test_roofline_skips_launch_bound_finalize_kernels():
    """A BN finalize (class 4 or 5) with the largest summed time does not
    become the roofline kernel: it is launch-latency bound, and the kernel with
    the most time among the others is taken (only finalizes: the largest)."""
    kernels = [("conv", 0, 12, 2.0, 1e9, 6.0e8), ("fin", 4, 36, 3.0, 0.0, 5.0e6),
               ("bfin", 5, 18, 1.0, 0.0, 2.0e6)]
    rl = bench.roofline(kernels, "bf16")
    assert rl["kernel"] == "conv"
    rl = bench.roofline([("fin", 4, 36, 3.0, 0.0, 5.0e6), ("bfin", 5, 18, 1.0, 0.0, 2.0e6)], "bf16")
    assert rl["kernel"] == "fin"
