"""The device fp64 exp / log(1 + x) / logistic functions of the task
kernels, compiled for the host and checked against the C library: worst
errors of a few units in the last place over their ranges, exact special
values.  (CPU only; the GPU parity tests check the kernels that use them.)"""
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(os.path.dirname(HERE), "paper_2206_00470_amd", "csrc")


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("fp64math") / "check")
    subprocess.check_call(["g++", "-O2", "-std=c++17", "-ffp-contract=off", "-I", CSRC, "-o", exe,
                           os.path.join(HERE, "fp64math_check.cpp")])
    return exe


def test_fp64math_against_the_c_library(checker):
    out = subprocess.check_output([checker, "2000000"], text=True).split("\n")
    worst = dict(zip(out[0].split()[0::2], map(float, out[0].split()[1::2])))
    assert worst["exp"] <= 2 and worst["log1p"] <= 4, worst
    assert worst["sigmoid"] <= 3 and worst["softplus"] <= 6, worst
    special = [float(v) for v in out[1].split()[1:]]
    # e^0 = 1, e^-746 underflows to 0, log(1 + 0) = 0, sigmoid(0) = 1/2, softplus(0) = log 2
    assert special[:4] == [1.0, 0.0, 0.0, 0.5]
    assert special[4] == pytest.approx(0.6931471805599453, rel=0, abs=4e-16)
