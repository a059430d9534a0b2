"""bench.py's command line on the CPU: more than one GPU is refused with a
message before anything touches a device, and the help lists every mode."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _run(*args):
    return subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                          timeout=120, env={**os.environ, "WORLD_SIZE": "1"})


def test_more_than_one_gpu_is_refused():
    r = _run("--gpus", "2")
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr


def test_help_lists_the_modes():
    r = _run("--help")
    assert r.returncode == 0
    for mode in ("bench", "counters", "decode_counters", "decode_split", "decode_sq", "gsweep", "layers", "summarize"):
        assert mode in r.stdout, mode


def test_timing_event_failure_is_an_exception_the_bench_catches():
    """Without a usable device, creating a fence-free timing event raises one of
    the exceptions the timed loop falls back on (torch's events) instead of
    crashing.  Run in a child process so the HIP runtime probe stays out of the
    test process."""
    code = (f"import sys; sys.path.insert(0, {ROOT!r}); import bench\n"
            "try:\n"
            "    bench.TimingEvent()\n"
            "    print('created')\n"
            "except (OSError, AttributeError, RuntimeError) as e:\n"
            "    print('refused', type(e).__name__)\n")
    try:
        import torch
        if torch.cuda.is_available():
            import pytest
            pytest.skip("a GPU is visible")
    except ImportError:
        pass
    r = subprocess.run([sys.executable, "-c", code], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    assert r.stdout.strip().startswith("refused"), r.stdout
