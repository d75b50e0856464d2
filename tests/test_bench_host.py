"""Host-side checks of bench.py that need no GPU: it measures one GPU only and
refuses to pretend otherwise."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, env=env, timeout=120)


def test_more_than_one_gpu_is_refused():
    r = _run(["--gpus", "2"])
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_a_distributed_launch_is_refused():
    r = _run([], {"WORLD_SIZE": "4"})
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_traffic_figures_come_from_the_counter_summaries():
    # every committed summary listed holds its per-launch traffic, the same
    # run's algorithmic bytes and the digests of the inject's sources; a
    # figure is reported only while those sources hash as recorded (else
    # None), and then lies within 2% of that run's algorithmic bytes
    import hashlib
    import re
    sys.path.insert(0, ROOT)
    import bench
    csrc = os.path.join(ROOT, "paper_2607_27090_amd", "csrc")
    for (workload, fused), (fname, key) in bench.TRAFFIC_PROFILES.items():
        path = os.path.join(ROOT, "profiles", fname)
        if not os.path.exists(path):
            assert bench.measured_traffic(workload, fused) is None
            continue
        text = open(path).read()
        assert re.search(rf"^{key}: \d+$", text, re.M), (fname, key)
        assert re.search(r"^algorithmic_bytes_per_launch: \d+$", text, re.M), fname
        want = dict(re.findall(r"(\S+\.h\w*) ([0-9a-f]{64})", text))
        assert set(want) == {"abi.hip", "common.hpp", "inject.hip", "launch.hpp"}, fname
        current = all(hashlib.sha256(open(os.path.join(csrc, n), "rb").read()).hexdigest() == d
                      for n, d in want.items())
        tb = bench.measured_traffic(workload, fused)
        assert (tb is not None) == current, (workload, fused)
        if tb is not None:
            assert 0.99 < tb["ratio"] < 1.02, (workload, fused, tb)
    assert bench.measured_traffic("tiny", True) is None


def _fake_rocprof(tmp, counter, inject_kib, copy_kib, n_inject):
    import csv
    d = tmp / counter
    (d / "host" / "1").mkdir(parents=True)
    with open(d / "host" / "1" / "run_counter_collection.csv", "w", newline="") as f:
        wr = csv.writer(f)
        wr.writerow(["Dispatch_Id", "Kernel_Name", "Counter_Name", "Counter_Value"])
        for i in range(n_inject):
            wr.writerow([i, "void is::inject_kernel<false, true>(int const*, long)", counter,
                         inject_kib[i % len(inject_kib)]])
        for i in range(3):
            wr.writerow([100 + i, "void is::stream_copy_kernel(unsigned int const*)", counter,
                         copy_kib])
        wr.writerow([200, "void at::native::fill(int)", counter, 5.0])
    (d / "bench.json").write_text("setup line\n" + json.dumps({
        "profile_pass": True, "workload": "llama3.1-8b", "k": 50, "nq": 1, "path": "fused",
        "kernel": "inject_kernel<false, true>", "inject_dispatches": n_inject,
        "algorithmic_bytes_per_launch": 524_288_000}) + "\n")
    return str(d)


def test_traffic_summary_scales_by_the_calibration_copy(tmp_path):
    # FETCH_SIZE reads half of what moves (the copy's 1 GiB as 512 MiB),
    # WRITE_SIZE all of it: the summary scales each by its own calibration
    f = _fake_rocprof(tmp_path, "FETCH_SIZE", [128000.0, 128000.0], 524288.0, 4)
    w = _fake_rocprof(tmp_path, "WRITE_SIZE", [256000.0], 1048576.0, 4)
    r = _run(["--summarize-traffic", f, w, "--title", "t", "--cmd", "rocprofv3 ... (fake)"])
    assert r.returncode == 0, r.stderr
    out = r.stdout
    total = 128000.0 * 1024 * 2 + 256000.0 * 1024
    assert f"traffic_bytes_per_launch: {round(total)}" in out
    assert "algorithmic_bytes_per_launch: 524288000" in out
    assert f"ratio {total / 524_288_000:.4f}" in out
    assert "inject.hip" in out and "rocprofv3 ... (fake)" in out


def test_traffic_summary_refuses_a_dispatch_count_mismatch(tmp_path):
    f = _fake_rocprof(tmp_path, "FETCH_SIZE", [1.0], 524288.0, 5)
    w = _fake_rocprof(tmp_path, "WRITE_SIZE", [1.0], 1048576.0, 4)
    meta = json.loads(open(os.path.join(f, "bench.json")).read().splitlines()[-1])
    meta["inject_dispatches"] = 4
    with open(os.path.join(f, "bench.json"), "w") as fh:
        fh.write(json.dumps(meta) + "\n")
    r = _run(["--summarize-traffic", f, w])
    assert r.returncode != 0 and "dispatches" in (r.stderr + r.stdout)


def test_stats_summary_lists_the_library_kernels(tmp_path):
    import csv
    d = tmp_path / "st"
    d.mkdir()
    with open(d / "run_kernel_stats.csv", "w", newline="") as fh:
        wr = csv.writer(fh)
        wr.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs",
                     "MaxNs", "StdDev"])
        wr.writerow(["void is::inject_kernel<false, true>(int)", 10, 1050000, 105000.0, 80.0,
                     100000, 110000, 1.0])
        wr.writerow(["void at::native::fill(int)", 3, 30000, 10000.0, 20.0, 9000, 11000, 1.0])
    (d / "bench.json").write_text(json.dumps({"value": 120.0, "unit": "us/request",
                                              "inject_launch_us": 104.8,
                                              "roofline": {"achieved": 5017.0, "frac": 0.627,
                                                           "peak": 8000.0}}) + "\n")
    r = _run(["--summarize-stats", str(d), "--title", "stats", "--cmd", "rocprofv3 x"])
    assert r.returncode == 0, r.stderr
    assert "| `is::inject_kernel<false, true>` | 10 | 105.00 |" in r.stdout
    assert "at::native" not in r.stdout
    assert "inject launch 104.8 us" in r.stdout


def test_stats_summary_includes_named_kernels_and_the_library_gemm(tmp_path):
    import csv
    d = tmp_path / "st"
    d.mkdir()
    long_name = "Cijk_Ailk_Bljk_BBS_BH_Bias_HA_S_SAV_UserArgs_MT256x256x64_MI16x16x1_SN_LDSB1_AFC1_AFEM1_ETC"
    with open(d / "run_kernel_stats.csv", "w", newline="") as fh:
        wr = csv.writer(fh)
        wr.writerow(["Name", "Calls", "TotalDurationNs", "AverageNs", "Percentage", "MinNs",
                     "MaxNs", "StdDev"])
        wr.writerow(["void is::scan_mfma_kernel<true>(int)", 5, 3000000, 600000.0, 60.0,
                     590000, 610000, 1.0])
        wr.writerow([long_name, 4, 2880000, 720000.0, 40.0, 700000, 740000, 1.0])
        wr.writerow(["void at::native::fill(int)", 3, 30000, 10000.0, 1.0, 9000, 11000, 1.0])
    (d / "bench.json").write_text(json.dumps({
        "value": 200.0, "unit": "us/request", "inject_launch_us": 12000.0,
        "roofline": {"achieved": 5000.0, "frac": 0.625, "peak": 8000.0},
        "library_gemm": {"what": "torch.matmul(...)", "us_median": 814.4, "TFLOPs": 643.8,
                         "bank_GBps": 2514.8}}) + "\n")
    r = _run(["--summarize-stats", str(d), "--include", "Cijk", "--title", "t", "--cmd", "x"])
    assert r.returncode == 0, r.stderr
    assert "| `is::scan_mfma_kernel<true>` | 5 | 600.00 |" in r.stdout
    # names past 90 characters are cut with an ellipsis
    assert f"| `{long_name[:87]}...` | 4 | 720.00 |" in r.stdout
    assert "at::native" not in r.stdout
    assert "814.4 us event-timed median, 643.8 TFLOP/s" in r.stdout
