"""bench.py's command line (CPU): one GPU only, and the options the driver and the profile commands use."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    r = run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_options_of_the_contract_and_the_profiles():
    r = run("--help")
    assert r.returncode == 0
    for opt in ("--gpus", "--steps", "--warmup", "--cpu-seconds", "--fused-steps", "--logp-steps", "--shard-steps",
                "--skip-logits", "--token-block", "--fused-schedule", "--copy-calibration"):
        assert opt in r.stdout, opt
