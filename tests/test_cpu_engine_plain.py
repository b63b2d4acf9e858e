"""The CPU engine's plain (non-vector) loops against the oracle: the same
cases as test_cpu_engine, in a child process with WSK_CPU_ENGINE=plain (the
choice is made once per process)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_cpu_engine_plain_loops():
    env = dict(os.environ, WSK_CPU_ENGINE="plain")
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_cpu_engine.py"), "-k", "gqa or mla"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-3000:] + r.stderr[-2000:]
