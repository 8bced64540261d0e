"""bench.py's command-line contract on the CPU: more than one GPU is refused
with a message before anything touches a GPU, and inconsistent window flags
are rejected."""
import subprocess
import sys
from pathlib import Path

ROOT = Path(__file__).resolve().parent.parent


def _run(*args):
    return subprocess.run([sys.executable, str(ROOT / "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, cwd=str(ROOT))


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_window_flags_are_checked():
    r = _run("--down", "9")
    assert r.returncode == 2 and "--down and --up" in r.stderr
    r = _run("--window", "4", "--down", "9", "--up", "6")
    assert r.returncode == 2
