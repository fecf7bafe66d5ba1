"""The register top-k network of blocks of four, compiled for the host.

The streaming selection residual_select4 runs per lane is plain C++; here it
is built with g++ and checked against numpy's lexsort (key descending, code
position ascending) on random and tie-heavy keys.
"""
import os
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC4 = os.path.join(HERE, "host", "topk4_driver.cpp")


def _expected(keys, k):
    c = np.broadcast_to(np.arange(keys.shape[1]), keys.shape)
    order = np.lexsort((c, -keys.astype(np.int64)), axis=-1)
    return np.sort(order[:, :k], axis=-1)


@pytest.fixture(scope="module")
def driver4(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("net4") / "topk4_driver")
    subprocess.run(["g++", "-O1", "-std=c++17", SRC4, "-o", exe], check=True)
    return exe


@pytest.mark.parametrize("D,RS,k", [(64, 16, 16), (64, 16, 1), (64, 32, 20), (64, 64, 64), (128, 16, 16),
                                    (128, 16, 5), (128, 32, 32), (128, 64, 40), (128, 128, 128), (128, 128, 97)])
def test_streaming_network_matches_sort(driver4, D, RS, k):
    """Blocks of four: 3D keys in code order, k largest with ties to the lower position."""
    rng = np.random.default_rng(D * 1000 + RS * 10 + k)
    rows = [np.abs(rng.standard_normal((150, 3 * D)).astype(np.float32)).view(np.uint32),
            rng.integers(0, 3, size=(150, 3 * D)).astype(np.uint32),
            np.zeros((3, 3 * D), np.uint32), np.full((2, 3 * D), 0x7F7FFFFF, np.uint32)]
    keys = np.concatenate(rows)
    inp = f"{D} {RS} {k} {keys.shape[0]}\n" + "\n".join(" ".join(map(str, r)) for r in keys.tolist())
    out = subprocess.run([driver4], input=inp, capture_output=True, text=True, check=True).stdout
    got = np.array([[int(x) for x in line.split()] for line in out.strip().splitlines()])
    np.testing.assert_array_equal(got, _expected(keys, k))
