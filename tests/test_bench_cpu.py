"""bench.py's host-side contract: one GPU only (more is refused before any device work, with
exit status 2), and its options parse."""
import os
import subprocess
import sys

REPO = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run_bench(*args):
    return subprocess.run([sys.executable, os.path.join(REPO, "bench.py"), *args], cwd=REPO,
                          capture_output=True, text=True, timeout=120)


def test_more_than_one_gpu_is_refused():
    res = run_bench("--gpus", "2")
    assert res.returncode == 2
    assert "one GPU only" in res.stdout + res.stderr


def test_options_parse():
    res = run_bench("--help")
    assert res.returncode == 0
    for opt in ("--steps", "--warmup", "--config", "--cpu-seconds", "--phase-sweeps",
                "--heldout-share", "--weighted", "--gibbs", "--tensor", "--bptf"):
        assert opt in res.stdout
