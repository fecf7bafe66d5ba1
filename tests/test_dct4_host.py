"""The DCT-II(4) butterfly of the HIP path (csrc/dct4.h), built for the host
with g++ and no contraction, against the oracle's float64 ranking keys of
blocks of four: the fp32 keys must stay within the rounding bound derived
below, the band in which the GPU parity tests accept either order."""
import os
import subprocess

import numpy as np

import oracle as O

HERE = os.path.dirname(os.path.abspath(__file__))

DCT4 = os.path.join(HERE, "host", "dct4_driver.cpp")


def test_dct4_butterfly_within_its_bound_of_the_oracle_keys(tmp_path):
    """The ranking keys of blocks of four: the HIP path's fp32 butterfly, built for the host
    without contraction, against the oracle's float64 |Z_j| (Eq. 1).  Error bound of the
    butterfly, u = 2^-24, M = max_n |x_n| of the channel: Z_1 = a (x0 - x3) + b (x1 - x2)
    with a, b the fp32 roundings of F_4[1][0], F_4[1][1] carries at most three roundings
    on each product term plus one on the sum, 4u (|F_4[1][0]| + |F_4[1][1]|) 2M = 7.4u M;
    Z_3 alike; Z_2 = ((x0 + x3) - (x1 + x2)) / 2 at most 4u M.  So |key32 - key64| <= 8u M
    = 2^-21 M, which the GPU parity tests use as the near-tie band of blocks of four."""
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
    k32 = (got & np.uint32(0x7FFFFFFF)).view(np.float32).astype(np.float64)      # [N][3]
    k64 = O.residual_keys_dct4(X.astype(np.float64)[:, :, None])[:, 0, :]      # [N][3] |Z| in float64
    M = np.abs(X.astype(np.float64)).max(axis=0)[:, None]
    err = np.abs(k32 - k64)
    assert np.all(err <= 2.0 ** -21 * M)
    assert err.max() > 0                    # the fp32 butterfly does round
    # integer inputs: every step is exact in fp32 except the products with a and b
    ints = slice(6000, 6500)
    np.testing.assert_array_equal(k32[ints, 1], k64[ints, 1])      # Z_2 of integers is exact
