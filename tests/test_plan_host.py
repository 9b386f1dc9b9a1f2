"""CPU: the launch planning (decode partition and workspace slots, the
prefill's XCD-aware work order, the automatic key-split count) at several
machine shapes, through a small C++ harness built with g++ against the
library's planning header."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "plan_harness.cpp")


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("plan") / "plan_harness")
    subprocess.run(["g++", "-O2", "-std=c++17", "-Wall", "-Werror", SRC, "-o", exe], check=True)
    return exe


@pytest.mark.parametrize("cus,xcds", [(32, 4), (64, 8), (256, 8), (256, 1), (80, 1)])
def test_partition_arithmetic(harness, cus, xcds):
    res = subprocess.run([harness, str(cus), str(xcds)], capture_output=True, text=True)
    assert res.returncode == 0 and res.stdout.startswith("ok"), res.stdout + res.stderr
