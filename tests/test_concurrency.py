"""Concurrent calls through the C ABI from several host threads and streams
give the bits of a single-thread call (the launch shape, and so the order of
every sum, depends only on the arguments and the device)."""
import os
import subprocess
import sys

import pytest
import torch

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_eight_threads_eight_streams_bit_identical():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    script = os.path.join(ROOT, "tests", "concurrent_spmm.py")
    env = dict(os.environ, PYTHONPATH=ROOT + os.pathsep + os.environ.get("PYTHONPATH", ""))
    r = subprocess.run([sys.executable, "-u", script], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=300)
    print(r.stdout, r.stderr)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-2000:]
    assert "all identical" in r.stdout
