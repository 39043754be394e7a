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
