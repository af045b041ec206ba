"""Host code under sanitizers: the planner with AddressSanitizer and
UndefinedBehaviorSanitizer (random valid and invalid tables, every getter,
structural invariants), and the host copy pool with ThreadSanitizer."""
import os
import subprocess

import sanitize


def _bin(path):
    if not os.path.exists(path):
        sanitize.build()
    return path


def test_planner_asan_ubsan():
    r = subprocess.run([_bin(sanitize.PLAN_BIN), "3000"], capture_output=True, text=True,
                       timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("OK"), r.stdout
    plans = int(r.stdout.split("plans=")[1].split()[0])
    assert plans > 12000  # most tables are valid and fully checked


def test_copy_pool_tsan():
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([_bin(sanitize.POOL_BIN)], capture_output=True, text=True, timeout=600,
                       env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "OK"
