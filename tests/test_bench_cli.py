"""bench.py's contract on the CPU: it refuses more than one GPU with a message, and its
CPU-only studies (the coordinator across instances, the local-policy ablation) run on
the scheduler-only executor and print one JSON document."""
import json
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args, timeout=600):
    return subprocess.run([sys.executable, "bench.py", *args], cwd=ROOT, capture_output=True, text=True,
                          timeout=timeout)


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode != 0
    assert "one GPU" in r.stderr


def test_policy_ablation_small_replay_prints_json():
    from ._lib import ensure_built
    ensure_built()
    r = _run("--policy-ablation", "--n-workflows", "12")
    assert r.returncode == 0, r.stderr[-2000:]
    out = json.loads(r.stdout.strip().splitlines()[-1])
    assert out["workflows"] == 12 and len(out["scenarios"]) >= 5
    for row in out["scenarios"]:
        for pol in ("pq", "fcfs", "llf"):
            assert 0.0 <= row[pol]["slo_attainment"] <= 1.0
            assert row[pol]["finished"] == 12
