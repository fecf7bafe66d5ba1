"""The seeded generator: reproducible substreams and the workload recipe."""
import math

import numpy as np

from synth import WORKLOADS, gen, scaled


def test_segments_reproducible_and_independent_of_order():
    w = scaled(WORKLOADS["llama8b"], seq_lens=(300,), n_layers=4)
    a = gen.segment(w, 0, 1, 3)
    b = gen.segment(w, 0, 1, 3)
    np.testing.assert_array_equal(a[0], b[0])
    np.testing.assert_array_equal(a[1], b[1])
    c = gen.segment(w, 0, 1, 2)
    assert not np.array_equal(a[0], c[0])
    K, V = gen.layer_cache(w, 0, threads=4)
    np.testing.assert_array_equal(K[2:4, 3], a[0])
    np.testing.assert_array_equal(V[2:4, 3], a[1])


def test_bf16_values_are_representable():
    w = scaled(WORKLOADS["llama8b"], seq_lens=(64,), n_layers=2)
    K, V, _ = gen.segment(w, 0, 0, 0)
    for x in (K, V):
        assert (x.view(np.uint32) & 0xFFFF == 0).all()
    q = gen.decode_queries(w, 0)
    assert (q.view(np.uint32) & 0xFFFF == 0).all()


def test_round_bf16_ties_to_even():
    x = np.array([1.00390625, 1.01171875, -1.00390625], np.float32)
    np.testing.assert_array_equal(gen.round_bf16_f32(x), np.array([1.0, 1.015625, -1.0], np.float32))


def test_correlation_and_needles():
    w = scaled(WORKLOADS["llama8b"], seq_lens=(8192,), n_layers=2)
    K, V, info = gen.segment(w, 0, 0, 5)
    rho = info["rho"]
    assert 0.75 <= rho <= 0.95
    mask = np.ones(K.shape[1], bool)
    mask[[p for p, _, _ in info["needles"]]] = False
    emp = np.corrcoef(K[0][mask].ravel(), K[1][mask].ravel())[0, 1]
    assert abs(emp - rho) < 0.01
    assert len(info["needles"]) == 16
    for pos, layer, ch in info["needles"]:
        assert len(set(ch.tolist())) == 16
        # the spiked channels carry the +5 offset on top of unit-variance noise
        assert K[layer, pos, ch].mean() > 2.0


def test_fixed_mode_mix():
    w = WORKLOADS["llama8b"]
    m = gen.fixed_modes(w)
    assert m.shape == (16, 8)
    assert np.bincount(m.ravel(), minlength=3).tolist() == [64, 45, 19]
    assert gen.fixed_modes(WORKLOADS["tiny"]).ravel().tolist() == [0, 1, 1, 2]
    m70 = gen.fixed_modes(WORKLOADS["long70b"])
    assert np.bincount(m70.ravel(), minlength=3).tolist() == [128, 128, 64]


def test_ragged_lengths():
    w = WORKLOADS["batched8b"]
    assert w.batch == 16
    assert all(4096 <= t <= 16384 for t in w.seq_lens)
    assert len(set(w.seq_lens)) > 8


def test_query_scale():
    w = WORKLOADS["llama8b"]
    q = gen.decode_queries(w, 3)
    assert q.shape == (32, 1, 32, 128)
    assert abs(np.mean(np.sum(q.astype(np.float64) ** 2, -1)) - 1.0) < 0.05
    p = gen.probe_queries(scaled(w, n_layers=2))
    assert p.shape == (2, 32, 256, 128)
    assert abs(p.std() * math.sqrt(128) - 1.0) < 0.01


def test_block_of_four_segments():
    w = scaled(WORKLOADS["llama8b_mixed"], n_layers=12, n_kv_heads=2, seq_lens=(3000,), n_needles=3)
    assert w.block_sizes == (2, 2, 4, 2, 2) and w.blocks[2] == (4, 4) and w.n_blocks == 5
    K, V, info = gen.block_segment(w, 0, 2, 1)
    K2, V2, _ = gen.block_segment(w, 0, 2, 1)
    assert K.shape == (4, 3000, 128) and np.array_equal(K, K2) and np.array_equal(V, V2)
    assert np.array_equal(K, gen.to_storage(K, w.dtype))            # bf16 values
    # first-order chain along depth: adjacent layers correlate by rho, layers two apart by rho^2
    mask = np.ones(3000, bool)
    mask[[p for p, _, _ in info["needles"]]] = False
    c01 = np.corrcoef(K[0, mask].ravel(), K[1, mask].ravel())[0, 1]
    c02 = np.corrcoef(K[0, mask].ravel(), K[2, mask].ravel())[0, 1]
    rho = info["rho"]
    assert abs(c01 - rho) < 0.01 and abs(c02 - rho * rho) < 0.01
    # pairs of the mixed schedule are the pair recipe's segments
    Kp, _, _ = gen.segment(w, 0, 5, 0)
    Kb, _, _ = gen.block_segment(w, 0, 4, 0)
    assert np.array_equal(Kp, Kb)
    Kfull, _ = gen.layer_cache(w, 0)
    assert np.array_equal(Kfull[4:8, 1], K)
    m = gen.fixed_modes(w)
    assert m.shape == (5, 2)
