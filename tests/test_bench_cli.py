"""bench.py's command-line contract on a host without a GPU: asking for more
than one GPU ends at once with a message and a nonzero status."""
import os
import subprocess
import sys

from tests.conftest import ROOT


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU only" in (r.stdout + r.stderr)


def test_gpu_process_check_skipped_under_a_profiler(monkeypatch):
    """Under rocprofv3 (ROCPROF* variables set) the bench does not start the
    amd-smi check: the profiler's preloaded library would start the GPU in the
    child, which then replaces itself through its "#!" line."""
    import subprocess as sp

    sys.path.insert(0, ROOT)
    import bench

    calls = []
    monkeypatch.setattr(sp, "run", lambda *a, **k: calls.append(a) or None)
    monkeypatch.setenv("ROCPROF_KERNEL_TRACE", "1")
    assert bench.gpu_processes() is None
    assert calls == []
