"""The DCT-II(4) butterfly of the HIP path (csrc/dct4.h), built for the host
with g++ and no contraction, against the oracle's float32 ranking keys of
blocks of four: the two sides must take the same top-k decisions, so the
keys must agree bit for bit."""
import os
import subprocess

import numpy as np

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))

DCT4 = os.path.join(HERE, "host", "dct4_driver.cpp")


def test_dct4_butterfly_matches_oracle_keys(tmp_path):
    """The ranking keys of blocks of four: the HIP path's fp32 butterfly, built for the host
    without contraction, equals the oracle's float32 evaluation bit for bit."""
    exe = str(tmp_path / "dct4_driver")
    subprocess.run(["g++", "-O2", "-ffp-contract=off", "-std=c++17", DCT4, "-o", exe], check=True)
    rng = np.random.default_rng(31)
    X = np.concatenate([
        O.round_bf16(rng.standard_normal((4, 3000)) * 4).astype(np.float32),
        rng.standard_normal((4, 3000)).astype(np.float32) * np.float32(1e3),
        rng.integers(-3, 4, size=(4, 500)).astype(np.float32),
    ], axis=1)
    inp = "\n".join(" ".join(str(int(v)) for v in row) for row in X.T.view(np.uint32).tolist())
    out = subprocess.run([exe], input=inp, capture_output=True, text=True, check=True).stdout
    got = np.array([[int(v) for v in line.split()] for line in out.strip().splitlines()], dtype=np.uint32)
    keys = O.residual_keys_dct4(X[:, :, None])[:, 0, :]          # [N][3] |Z| in float32
    np.testing.assert_array_equal(got & np.uint32(0x7FFFFFFF), keys.view(np.uint32))
