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


def test_power_of_two_scale_of_every_amax_matches_the_oracle(tmp_path):
    """The kernels' power-of-two scale (quant_math.hpp on the host) for every finite
    bf16 amax equals the oracle's 2^k, and the multiplier is exactly 2^-k."""
    import numpy as np
    from oracle import quant, ue8m0
    exe = str(tmp_path / "pow2_scale_dump")
    subprocess.run(["g++", "-O2", "-std=c++17", f"-I{INC}", os.path.join(ROOT, "tests", "host", "pow2_scale_dump.cpp"),
                    "-o", exe], check=True)
    out = subprocess.run([exe], capture_output=True, text=True, check=True, timeout=120).stdout
    rows = np.array([ln.split() for ln in out.splitlines()], dtype=np.uint64).astype(np.uint32)
    amax = quant.bf16_bits_to_f32(rows[:, 0].astype(np.uint16)).astype(np.float64)
    k = ue8m0.scale_exponent(amax)
    assert np.array_equal(rows[:, 1].view(np.float32).astype(np.float64), np.ldexp(1.0, k))
    assert np.array_equal(rows[:, 2].view(np.float32).astype(np.float64), np.ldexp(1.0, -k))
