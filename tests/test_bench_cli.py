"""bench.py on the CPU: its command line, the bytes it counts per step, and
the counter-summary names it reads (no GPU needed)."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                          capture_output=True, text=True, timeout=120)


def test_help():
    r = _run("--help")
    assert r.returncode == 0 and "--no-probe" in r.stdout and "--plan" in r.stdout


@pytest.mark.parametrize("n", ["2", "8"])
def test_more_than_one_gpu_is_refused_with_a_message(n):
    r = _run("--gpus", n)
    assert r.returncode == 2 and "one GPU" in r.stderr


def test_algorithmic_bytes_per_mode():
    n = 1000
    bench.K, bench.E_G = 16, 2
    ags = bench.algorithmic_bytes(n, "ags")
    assert ags == {"step": 48 * n, "finalize": 0, "second_pass": 0, "whole_step": 48 * n}
    assert bench.algorithmic_bytes(n, "ags", elementwise=True)["step"] == 56 * n
    lars = bench.algorithmic_bytes(n, "lars", reuse_w_norms=False)
    # first pass: replicas + w read, mean written; second: mean, w, m read, w, m written
    assert lars["step"] == (32 + 4 + 4) * n and lars["second_pass"] == (4 + 16) * n
    assert lars["whole_step"] == 48 * n
    # with the weight norms carried from the update pass the first pass skips w
    assert bench.algorithmic_bytes(n, "lars")["step"] == (32 + 4) * n
    bench.K, bench.E_G = 2, 2      # K e_g <= 8: the second pass re-reads the replicas
    lars = bench.algorithmic_bytes(n, "lars", reuse_w_norms=False)
    assert lars["step"] == (4 + 4) * n and lars["second_pass"] == (4 + 16) * n
    bench.K, bench.E_G = 16, 2


def test_counter_summary_names():
    w = "resnet50_k16_bf16"
    assert bench.workload_key(w, False) == w
    assert bench.workload_key(w, False, "global", "sgd") == w      # same step kernel as AGS
    assert bench.workload_key(w, False, "global", "static") == w
    assert bench.workload_key(w, False, "global", "lars") == w + "_lars"
    assert bench.workload_key(w, True) == w + "_elementwise"
    assert bench.workload_key(w, False, "layer") == w + "_layer_delta"


def test_traffic_is_null_for_a_missing_summary():
    assert bench.read_traffic("no_such_workload", "step") is None
