"""bench.py's command-line contract on the CPU: more than one GPU (by flag or
by a torch.distributed WORLD_SIZE) is refused with exit status 2 and a
message on stderr, before any GPU work and with nothing on stdout."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.parametrize("args,env", [(["--gpus", "2"], {}), (["--gpus", "8"], {}), ([], {"WORLD_SIZE": "2"})])
def test_more_than_one_gpu_is_refused(args, env):
    e = dict(os.environ, **env)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), *args], capture_output=True, text=True,
                       timeout=120, env=e, cwd=ROOT)
    assert r.returncode == 2, (r.returncode, r.stderr[-500:])
    assert "exactly one GPU" in r.stderr
    assert r.stdout.strip() == ""

