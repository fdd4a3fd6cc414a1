"""The allocating entry points under stream capture: in a fresh process the
first split-K call finds no workspace, so under capture it must return
KERNELARC_ERR_UNSUPPORTED (a clean error, nothing enqueued) and the eager
call afterwards must work.  The case runs in a child process of its own."""
import os
import subprocess
import sys

import pytest
import torch

pytestmark = pytest.mark.gpu

HERE = os.path.dirname(os.path.abspath(__file__))


def test_first_split_call_under_capture_is_refused():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    print("[gpu-case] capture: first split-K call in a fresh process", flush=True)
    r = subprocess.run([sys.executable, "-u", os.path.join(HERE, "capture_first_split_call.py")],
                       capture_output=True, text=True, timeout=300)
    print(r.stdout[-2000:])
    print(r.stderr[-2000:])
    assert r.returncode == 0, r.stderr[-2000:]
    assert "CAPTURE_OK" in r.stdout
