"""Host planners under random and malformed inputs, built with the host address and
undefined-behaviour sanitizers (CPU only; no device code is built or run)."""

import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2606_01065_amd", "csrc")


@pytest.fixture(scope="module")
def fuzz(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("plan_fuzz") / "plan_fuzz")
    cmd = [gxx, "-O1", "-g", "-std=c++17", "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-I" + os.path.join(ROOT, "include"), "-I" + CSRC,
           os.path.join(ROOT, "tests", "plan_fuzz.cpp"), os.path.join(CSRC, "plan.cpp"), "-o", exe]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        pytest.skip("host sanitizers not available: " + r.stderr[-300:])
    return exe


@pytest.mark.parametrize("seed", [21, 22, 23, 24])
def test_planners_survive_malformed_inputs(fuzz, seed):
    r = subprocess.run([fuzz, str(seed), "50000"], capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:] + r.stderr[-4000:]
    tag, ok, _, err = r.stdout.split()
    assert tag == "ok" and int(ok) > 1000 and int(err) > 1000
