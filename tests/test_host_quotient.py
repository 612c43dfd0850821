"""The kernels' per-element quotient (quant_math.hpp, compiled for the host with
g++) against plain IEEE fp32 division, over (x, amax) bf16 pairs: a sample of
amax values by default, every amax under the `slow` marker."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "host", "quotient_check.cpp")
INC = os.path.join(ROOT, "paper_2601_18150_amd", "csrc")


@pytest.fixture(scope="module")
def harness(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("host") / "quotient_check")
    subprocess.run(["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-fno-fast-math", f"-I{INC}", SRC, "-o", exe],
                   check=True)
    return exe


def test_quotient_equals_ieee_division_sampled_amax(harness):
    r = subprocess.run([harness, "61"], capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:]
    assert "mismatches 0" in r.stdout


@pytest.mark.slow
def test_quotient_equals_ieee_division_every_amax(harness):
    r = subprocess.run([harness, "1"], capture_output=True, text=True, timeout=3000)
    assert r.returncode == 0, r.stdout[-2000:]
