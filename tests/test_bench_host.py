"""Host-side checks of bench.py that need no GPU: it measures one GPU only and
refuses to pretend otherwise."""
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
    # every listed summary exists and holds its per-launch figure and source
    # hashes; a figure is reported only while the kernel sources hash as
    # recorded (else None), and then lies within 1% of the workload's
    # algorithmic bytes
    import hashlib
    import re
    sys.path.insert(0, ROOT)
    import bench
    algorithmic = {"llama8b": 524.68e6, "concurrency": 33.717e9, "llama70b": 29.398e9,
                   "retrieval1m": 65.605e9}
    csrc = os.path.join(ROOT, "paper_2607_27090_amd", "csrc")
    for (workload, fused), (fname, key) in bench.TRAFFIC_PROFILES.items():
        text = open(os.path.join(ROOT, "profiles", fname)).read()
        assert re.search(rf"^{key}: \d+$", text, re.M), (fname, key)
        want = dict(re.findall(r"(\S+\.h\w*) ([0-9a-f]{64})", text))
        assert set(want) == {"inject.hip", "common.hpp"}, fname
        current = all(hashlib.sha256(open(os.path.join(csrc, n), "rb").read()).hexdigest() == d
                      for n, d in want.items())
        tb = bench.measured_traffic(workload, fused)
        assert (tb is not None) == current, (workload, fused)
        if tb is not None:
            assert abs(tb / algorithmic[workload] - 1) < 0.01, (workload, fused, tb)
    assert bench.measured_traffic("tiny", True) is None
