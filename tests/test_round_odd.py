"""The kernels' fp64 -> bf16 rounding (fp64 pair arithmetic): a float rounded to odd from the fp64
value, then rounded to nearest-even bf16 as the hardware's conversion does, must equal the
oracle's single round-to-nearest-even of the fp64 value (no GPU).

tests/round_odd.cpp runs the library's own f32_round_odd (kparams.hpp) on the host; the
nearest-even float -> bf16 step is torch's, and the expected values come from the oracle's encode,
which tests/test_oracle_pins.py pins against torch and hand-made ties."""

import os
import shutil
import subprocess

import numpy as np
import pytest
import torch

from oracle import splice_oracle as O

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def round_odd(tmp_path_factory):
    gxx = shutil.which("g++")
    if gxx is None:
        pytest.skip("g++ not available")
    exe = str(tmp_path_factory.mktemp("round_odd") / "round_odd")
    subprocess.run([gxx, "-O2", "-std=c++20", "-Wall", "-Wextra", "-Werror", "-I" + os.path.join(ROOT, "include"),
                    "-I" + os.path.join(ROOT, "paper_2606_01065_amd", "csrc"),
                    os.path.join(ROOT, "tests", "round_odd.cpp"), "-o", exe], check=True)

    def run(x: np.ndarray) -> np.ndarray:
        text = "\n".join(f"{b:016x}" for b in np.asarray(x, dtype=np.float64).view(np.uint64).tolist())
        out = subprocess.run([exe], input=text, capture_output=True, text=True, check=True).stdout.split()
        return np.array([int(h, 16) for h in out], dtype=np.uint32).view(np.float32)
    return run


def _bf16_of_float(f: np.ndarray) -> np.ndarray:
    return torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def test_round_odd_then_nearest_even_is_one_rounding(round_odd):
    rng = np.random.default_rng(5)
    normal = rng.standard_normal(100000) * np.exp2(rng.integers(-20, 20, 100000))
    # values at and next to bf16 ties: a bf16 value plus half its spacing, nudged by a few fp64 ulps
    base = O.decode(O.encode(rng.standard_normal(20000), O.BF16), O.BF16)
    half = O.ulp(base, O.BF16) / 2
    nudge = rng.integers(-3, 4, 20000)
    ties = np.nextafter(base + half, np.where(nudge >= 0, np.inf, -np.inf))
    for _ in range(3):
        ties = np.where(nudge != 0, np.nextafter(ties, np.where(nudge > 0, np.inf, -np.inf)), base + half)
    exact_ties = base + half
    # float ties too (where a float nearest-even conversion alone would decide wrongly)
    fl = rng.standard_normal(20000).astype(np.float32).astype(np.float64)
    fl_ties = fl + np.ldexp(1.0, np.frexp(fl)[1] - 25) * rng.choice([-1, 1], 20000)
    tiny = rng.standard_normal(20000) * 1e-39                   # bf16 / f32 subnormals
    edge = np.array([0.0, -0.0, 1.0, -1.0, 2.0 ** -133, 2.0 ** -134, 3 * 2.0 ** -135, 1e-45, 3.3e38, -3.3e38])
    x = np.concatenate([normal, ties, exact_ties, fl_ties, tiny, edge])
    got = _bf16_of_float(round_odd(x))
    want = O.encode(x, O.BF16)
    bad = np.flatnonzero(got != want)
    assert bad.size == 0, [(float(x[i]), hex(got[i]), hex(want[i])) for i in bad[:5]]


def test_plain_nearest_even_float_would_double_round(round_odd):
    """The reason for rounding to odd: going through a nearest-even float first rounds some fp64
    values twice, and those come out one bf16 ulp off; rounding to odd does not."""
    x = np.array([1.0 + 2.0 ** -8 + 2.0 ** -30])        # just above a bf16 tie, below float resolution
    twice = _bf16_of_float(x.astype(np.float32))            # float rounds onto the tie, then ties to even
    assert twice[0] != O.encode(x, O.BF16)[0]
    assert _bf16_of_float(round_odd(x))[0] == O.encode(x, O.BF16)[0]
