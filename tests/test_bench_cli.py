"""bench.py's command line on a host without a GPU: a request for more than one GPU (by flag
or by a launcher's WORLD_SIZE) ends with exit status 2 and a message, before any GPU work."""
import os
import subprocess
import sys

BENCH = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "bench.py")


def _run(args, env_extra=None):
    env = dict(os.environ)
    env.update(env_extra or {})
    return subprocess.run([sys.executable, BENCH, *args], capture_output=True, text=True,
                          env=env, timeout=120)


def test_more_than_one_gpu_is_refused():
    for args, extra in ((["--gpus", "2"], None), (["--gpus", "8"], None),
                        ([], {"WORLD_SIZE": "4"})):
        r = _run(args, extra)
        assert r.returncode == 2, (args, r.returncode, r.stderr)
        assert "one GPU only" in r.stderr
        assert r.stdout == ""
