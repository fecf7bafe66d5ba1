"""The register top-k network of the HIP path, compiled for the host.

The selection routine the compress and probe kernels run per lane is plain
C++; here it is built with g++ and checked against numpy's lexsort (key
descending, channel ascending) on random and tie-heavy keys.
"""
import os
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "host", "topk_net_driver.cpp")


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    exe = str(tmp_path_factory.mktemp("net") / "topk_net_driver")
    subprocess.run(["g++", "-O1", "-std=c++17", SRC, "-o", exe], check=True)
    return exe


def _expected(keys, k):
    c = np.broadcast_to(np.arange(keys.shape[1]), keys.shape)
    order = np.lexsort((c, -keys.astype(np.int64)), axis=-1)
    return np.sort(order[:, :k], axis=-1)


@pytest.mark.parametrize("D,GS,k", [(64, 8, 8), (64, 8, 3), (64, 16, 16), (64, 16, 9), (64, 64, 64),
                                    (64, 64, 40), (128, 16, 16), (128, 16, 11), (128, 8, 1),
                                    (128, 128, 128), (128, 128, 77)])
def test_network_matches_sort(driver, D, GS, k):
    rng = np.random.default_rng(D * 1000 + GS * 10 + k)
    rows = []
    # float-like keys: |a - b| bit patterns of bf16-valued differences
    a = rng.standard_normal((200, D)).astype(np.float32)
    b = rng.standard_normal((200, D)).astype(np.float32)
    rows.append(np.abs(a - b).view(np.uint32))
    # heavy ties
    rows.append(rng.integers(0, 4, size=(200, D)).astype(np.uint32))
    rows.append(np.zeros((3, D), np.uint32))
    rows.append(np.full((3, D), 0x7F7FFFFF, np.uint32))
    keys = np.concatenate(rows)
    inp = f"{D} {GS} {k} {keys.shape[0]}\n" + "\n".join(" ".join(map(str, r)) for r in keys.tolist())
    out = subprocess.run([driver], input=inp, capture_output=True, text=True, check=True).stdout
    got = np.array([[int(x) for x in line.split()] for line in out.strip().splitlines()])
    np.testing.assert_array_equal(got, _expected(keys, k))
