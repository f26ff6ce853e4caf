"""The benchmark's command line on the CPU: it runs on one GPU only and says so for any other
count, and it names every configuration it can profile (no GPU is touched by these checks)."""
import subprocess
import sys
from pathlib import Path

ROOT = Path(__file__).resolve().parents[1]


def run(*args):
    return subprocess.run([sys.executable, str(ROOT / "bench.py"), *args], capture_output=True,
                          text=True, timeout=120, cwd=ROOT)


def test_more_than_one_gpu_is_refused_with_a_message():
    for n in ("2", "8"):
        r = run("--gpus", n)
        assert r.returncode == 2
        assert "one GPU only" in r.stderr and f"--gpus {n}" in r.stderr
        assert r.stdout == ""


def test_help_lists_the_profile_configurations():
    r = run("--help")
    assert r.returncode == 0
    for c in ("c0", "c2", "c3", "c3w", "c4", "f3", "f4"):
        assert c in r.stdout
