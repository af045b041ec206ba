"""Host-only sanitizer builds of the planner (ASan + UBSan), the host copy
pool (TSan), the reachability decision of the loads (ASan + UBSan, against
a fake memory map) and the per-tensor path's schedule (ASan + UBSan, carried
out on host buffers). Built with g++ from the library's own sources."""
from __future__ import annotations

import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
CSRC = os.path.join(ROOT, "paper_2607_18957_amd", "csrc")
INC = os.path.join(ROOT, "include")
PLAN_BIN = os.path.join(HERE, "plan_fuzz")
POOL_BIN = os.path.join(HERE, "pool_tsan")
REACH_BIN = os.path.join(HERE, "reach_check")
PERTENSOR_BIN = os.path.join(HERE, "pertensor_check")


def build() -> None:
    common = ["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-I", INC, "-I", CSRC]
    subprocess.check_call(common + ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                                    "-o", PLAN_BIN, os.path.join(HERE, "plan_fuzz.cpp"),
                                    os.path.join(CSRC, "plan.cpp")])
    subprocess.check_call(common + ["-fsanitize=thread", "-pthread", "-o", POOL_BIN,
                                    os.path.join(HERE, "pool_tsan.cpp")])
    subprocess.check_call(common + ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                                    "-o", REACH_BIN, os.path.join(HERE, "reach_check.cpp")])
    subprocess.check_call(common + ["-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                                    "-o", PERTENSOR_BIN, os.path.join(HERE, "pertensor_check.cpp")])
