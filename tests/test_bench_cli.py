"""bench.py's command-line contract and the committed traffic profiles (CPU)."""
import glob
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args],
                          capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_help_lists_the_measurement_modes():
    r = run("--help")
    assert r.returncode == 0
    for opt in ("--steps", "--warmup", "--surface", "--layer-surface", "--layer-dense", "--gemm-sweep",
                "--clock-sweep", "--next-profile", "--cpu-configs", "--score-ab"):
        assert opt in r.stdout, opt


def test_committed_traffic_matches_the_kernel_source():
    """roofline.traffic comes from the committed FETCH/WRITE profiles only
    while they were taken on the current attention source and flags: every
    workload's record carries the hash bench.py computes now."""
    sys.path.insert(0, ROOT)
    import importlib.util
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    bench = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(bench)
    h = bench.kernel_source_hash()
    files = sorted(glob.glob(os.path.join(ROOT, "profiles", "attn_kernel_*_traffic.json")))
    assert len(files) == 5
    for f in files:
        rec = json.load(open(f))
        assert rec["kernel_source_hash"] == h, f
        assert 1.0 <= rec["hbm_bytes_per_launch"] / rec["algorithmic_bytes_per_launch"] < 3.0
