"""bench.py as the driver runs it, on the CPU: the one-GPU limit is refused
with a message, and a run leaves no process behind (bench.py starts no
child process; the oracle baseline runs in-process)."""
import os
import signal
import subprocess
import sys

import psutil
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run_in_own_group(args, timeout=600):
    p = subprocess.Popen([sys.executable, os.path.join(ROOT, "bench.py"), *args], cwd=ROOT,
                         stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, start_new_session=True)
    try:
        out, _ = p.communicate(timeout=timeout)
    except subprocess.TimeoutExpired:
        os.killpg(p.pid, signal.SIGKILL)
        raise
    left = [q.pid for q in psutil.process_iter(["pid"]) if _pgid(q.pid) == p.pid]
    return p.returncode, out, left


def _pgid(pid):
    try:
        return os.getpgid(pid)
    except (ProcessLookupError, PermissionError):
        return None


def test_more_than_one_gpu_is_refused_and_nothing_is_left():
    rc, out, left = _run_in_own_group(["--gpus", "2"])
    assert rc != 0
    assert "one GPU" in out
    assert left == []


def test_run_without_a_gpu_fails_loudly_and_leaves_nothing():
    import torch
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    rc, out, left = _run_in_own_group(["--steps", "1", "--warmup", "1"])
    assert rc != 0
    assert left == []
