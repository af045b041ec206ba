"""Host code under sanitizers: the planner with AddressSanitizer and
UndefinedBehaviorSanitizer (random valid and invalid tables, every getter,
structural invariants), and the host copy pool with ThreadSanitizer."""
import os
import subprocess

import pytest

import sanitize


def _bin(path):
    if not os.path.exists(path):
        sanitize.build()
    return path


@pytest.mark.parametrize("groups_max,iters", [(None, 3000), ("64", 1000)],
                         ids=["default", "groups64"])
def test_planner_asan_ubsan(groups_max, iters):
    """The default planner, and one that moves every pinned chunk of up to 64
    run groups by group copies (so that the group layout check meets many
    groups per chunk)."""
    env = dict(os.environ)
    env.pop("II_PINNED_GROUPS_MAX", None)
    if groups_max:
        env["II_PINNED_GROUPS_MAX"] = groups_max
    r = subprocess.run([_bin(sanitize.PLAN_BIN), str(iters)], capture_output=True, text=True,
                       timeout=600, env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("OK"), r.stdout
    plans = int(r.stdout.split("plans=")[1].split()[0])
    assert plans > 4 * iters  # most tables are valid and fully checked


def test_copy_pool_tsan():
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1")
    r = subprocess.run([_bin(sanitize.POOL_BIN)], capture_output=True, text=True, timeout=600,
                       env=env)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "OK"


def test_reachability_decision():
    """reach.h on a fake memory map: a range is reachable only inside one
    device or pinned host allocation (not across two adjacent ones, not over
    a pageable hole, not one byte past the end), ranges packed in one arena
    cost one allocation query, and a later range that leaves the allocation
    found last is still caught."""
    r = subprocess.run([_bin(sanitize.REACH_BIN)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.strip() == "OK"


def test_pertensor_schedule():
    """The per-tensor path's host schedule (pertensor.h), which names every
    staging copy and host-to-device copy of ii_load_pertensor from a pageable
    blob: on the 100,000-tensor stress table with 16 MiB slots at depth 3,
    on slots smaller than the tensors and on 3,000 random tables (empty
    tensors, rows at a stride), every staging copy stays inside its slot and
    inside one row of its tensor, every device copy inside its slot and its
    tensor and only over bytes staged in the current fill of the slot, slots
    are handed over round robin, and carried out on host memory the
    destinations equal the tensors read straight from the blob."""
    r = subprocess.run([_bin(sanitize.PERTENSOR_BIN)], capture_output=True, text=True,
                       timeout=600)
    assert r.returncode == 0, r.stdout + r.stderr
    assert r.stdout.startswith("OK"), r.stdout
    assert int(r.stdout.split("copies=")[1]) >= 100_000
