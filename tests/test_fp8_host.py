"""The FP8 E4M3 encoder of the HIP path (csrc/fp8.h), built for the host with
g++ and checked against the oracle's rounding on float32 inputs: random
values, every exact midpoint of the E4M3 grid, subnormals, the saturation
range and signed zero."""
import os
import subprocess

import numpy as np
import pytest

import oracle as O
from gpu_cases import E4M3

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "host", "fp8_driver.cpp")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("fp8") / "fp8_driver")
    subprocess.run(["g++", "-O1", "-std=c++17", SRC, "-o", exe], check=True)
    return exe


def test_encoder_matches_oracle_rounding(driver):
    rng = np.random.default_rng(11)
    grid = np.sort(E4M3[:127])
    mids = ((grid[:-1] + grid[1:]) / 2).astype(np.float32)              # exact in float32
    xs = np.concatenate([
        rng.standard_normal(20000).astype(np.float32) * 2,
        rng.uniform(-600, 600, 5000).astype(np.float32),
        rng.uniform(-0.03, 0.03, 5000).astype(np.float32),
        mids, -mids, grid.astype(np.float32), -grid.astype(np.float32),
        np.array([448, 449, 464, 470, 479.9, 480, 1e9, -1e9, 2.0 ** -10, 3 * 2.0 ** -10,
                  2.0 ** -6, np.nextafter(np.float32(2.0 ** -6), np.float32(0)), 0.0, -0.0], np.float32),
    ]).astype(np.float32)
    inp = "\n".join(str(int(u)) for u in xs.view(np.uint32))
    out = subprocess.run([driver], input=inp, capture_output=True, text=True, check=True).stdout
    codes = np.array([int(v) for v in out.split()], dtype=np.int64)
    got = E4M3[codes]
    want = O.round_e4m3(xs.astype(np.float64))
    np.testing.assert_array_equal(got, want)
    # the sign survives on zero
    assert codes[-1] == 0x80 and codes[-2] == 0x00

