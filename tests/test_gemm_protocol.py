"""CPU check of the FP4 GEMM's LDS stage protocol (copy counts per wave, vmcnt waits, stage
reuse) for every configuration the kernel instantiates, using the kernel's own geometry and
copy assignment (paper_2607_26515_amd/csrc/gemm_geo.h) compiled for the host.  The same
check run on planted mistakes (a wait one copy short, a refill before the barrier, a padding
copy on an operand) must fail, so it is able to see them."""
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "gemm_protocol_check.cpp")


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("proto") / "gemm_protocol_check")
    r = subprocess.run(["g++", "-std=c++17", "-O1", "-Wall", "-I",
                        os.path.join(ROOT, "paper_2607_26515_amd", "csrc"), SRC, "-o", exe],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    return exe


def test_every_configuration_keeps_the_protocol(checker):
    r = subprocess.run([checker], capture_output=True, text=True, timeout=300)
    assert r.returncode == 0, r.stdout[-4000:]
    assert " configurations, 0 errors" in r.stdout


@pytest.mark.parametrize("plant,what", [(1, "complete"), (2, "before every wave is done reading"),
                                        (3, "written by 2 copies")])
def test_planted_mistakes_are_reported(checker, plant, what):
    r = subprocess.run([checker, str(plant)], capture_output=True, text=True, timeout=300)
    assert r.returncode == 1
    assert what in r.stdout
