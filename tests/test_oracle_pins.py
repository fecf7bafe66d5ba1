"""Pins of the CPU oracle against facts that do not come from the oracle itself.

Each test checks the oracle against a closed form, a textbook or library
routine, brute force on tiny inputs, an invariant of the method, or the
hand-worked example in ``tests/golden/worked_pair_d4.txt`` (derived by hand
from Eqs. (1)-(3) of the paper, Section 3).
"""
import itertools
import math
import os

import numpy as np
import pytest
import scipy.fft
import scipy.special

import oracle as O
from synth import WORKLOADS, gen, scaled

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_pair_d4.txt")


def _golden():
    vals = {}
    with open(GOLDEN) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            name, rest = line.split(":", 1)
            vals[name.strip()] = np.array([float(x) for x in rest.split()])
    return vals


# ---------------------------------------------------------------- Eq. (1)
@pytest.mark.parametrize("B", [2, 4, 8])
def test_dct_is_orthonormal(B):
    F = O.dct_matrix(B)
    np.testing.assert_allclose(F @ F.T, np.eye(B), atol=1e-14)


def test_dct2_is_haar():
    h = np.array([[1.0, 1.0], [1.0, -1.0]]) / np.sqrt(2.0)
    np.testing.assert_allclose(O.dct_matrix(2), h, atol=1e-16)


@pytest.mark.parametrize("B", [2, 4])
def test_factorize_matches_scipy_dct(B):
    rng = np.random.default_rng(1)
    X = rng.standard_normal((B, 7, 5))
    ref = scipy.fft.dct(X, type=2, norm="ortho", axis=0)
    np.testing.assert_allclose(O.depth_factorize(X), ref, atol=1e-13)


@pytest.mark.parametrize("B", [2, 4, 8])
def test_projectors_resolve_identity(B):
    P = O.dct_projectors(B)
    F = O.dct_matrix(B)
    for k in range(B):
        np.testing.assert_allclose(P[k], np.outer(F[k], F[k]), atol=1e-15)
    np.testing.assert_allclose(P.sum(0), np.eye(B), atol=1e-15)


def test_b2_projectors_exact_and_images_correctly_rounded():
    P = O.dct_projectors(2)
    np.testing.assert_array_equal(P, [[[0.5, 0.5], [0.5, 0.5]], [[0.5, -0.5], [-0.5, 0.5]]])
    # bf16 inputs whose mean sits exactly halfway between two bf16 values
    a = np.array([1.0, 1.0078125, -3.0, 2.0 ** -20])
    b = np.array([1.0078125, 1.0234375, -3.015625, 2.0 ** -20])
    X = np.stack([a, b])[:, None, :]
    unit = O.compress_unit(X, X, O.RESIDUAL, 4, "bf16")
    np.testing.assert_array_equal(unit["MK"][0], O.round_bf16((a + b) / 2))
    np.testing.assert_array_equal(np.sort(unit["VK"][0]), np.sort(O.round_bf16((a - b) / 2)))


def test_round_trip():
    rng = np.random.default_rng(2)
    X = rng.standard_normal((2, 33, 16))
    np.testing.assert_allclose(O.depth_reconstruct(O.depth_factorize(X)), X, atol=1e-14)


# ---------------------------------------------------------------- storage rounding
def test_round_bf16_against_bit_rounding():
    # float32 -> bf16 by integer round-to-nearest-even on the bit pattern (a
    # different construction), for inputs exactly representable in float32
    rng = np.random.default_rng(3)
    x = np.concatenate([rng.standard_normal(20000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 20000),
                        np.array([1.00390625, 1.01171875, -1.00390625, 0.0, -0.0, 1e-40, 3.3e38], np.float32)])
    x = x.astype(np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    r = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    ref = r.astype(np.uint32).view(np.float32).astype(np.float64)
    got = O.round_bf16(x.astype(np.float64))
    np.testing.assert_array_equal(got, ref)


# ---------------------------------------------------------------- residual channels
def _brute_topk(key, k):
    """All k-subsets: maximize the descending key vector, then the smallest index set."""
    d = len(key)
    best, best_set = None, None
    for sub in itertools.combinations(range(d), k):
        v = sorted((key[i] for i in sub), reverse=True)
        if best is None or v > best:
            best, best_set = v, sub
    # among all sets with that key multiset, lexicographically smallest indices
    cands = [s for s in itertools.combinations(range(d), k)
             if sorted((key[i] for i in s), reverse=True) == best]
    return sorted(min(cands))


@pytest.mark.parametrize("d,k", [(6, 2), (8, 3), (9, 4), (10, 5), (7, 7), (5, 1)])
def test_topk_brute_force(d, k):
    rng = np.random.default_rng(d * 100 + k)
    for trial in range(40):
        # small integers force many ties
        a = rng.integers(-3, 4, size=d).astype(np.float32)
        b = rng.integers(-3, 4, size=d).astype(np.float32)
        got = O.residual_channels(a[None], b[None], k)[0].tolist()
        key = np.abs(a - b).tolist()
        assert got == _brute_topk(key, k), (a, b)


def test_topk_key_is_float32():
    # a difference that float32 rounds: the key must tie, so the lower index wins
    a = np.array([1.0, 1.0], dtype=np.float32)
    b = np.array([np.float32(2.0 ** -25), 0.0], dtype=np.float32)
    # fl32(1 - 2^-25) = 1 exactly, so both keys are 1.0
    assert O.residual_channels(a[None], b[None], 1)[0].tolist() == [0]


def test_identical_layers_zero_residual():
    rng = np.random.default_rng(4)
    X = rng.standard_normal((11, 16)).astype(np.float32)
    unit = O.compress_unit(np.stack([X, X]), np.stack([X, X]), O.RESIDUAL, 5, "f32")
    np.testing.assert_array_equal(unit["VK"], 0.0)
    np.testing.assert_array_equal(unit["VV"], 0.0)
    np.testing.assert_array_equal(unit["IK"], np.tile(np.arange(5), (11, 1)))
    np.testing.assert_array_equal(unit["MK"], X.astype(np.float64))


def test_k_equals_d_reconstructs_exactly():
    rng = np.random.default_rng(5)
    d = 16
    K = rng.standard_normal((2, 9, d))
    V = rng.standard_normal((2, 9, d))
    unit = O.compress_unit(K, V, O.RESIDUAL, d, "f64")
    for par in (0, 1):
        np.testing.assert_allclose(O.reconstruct_layer(unit, O.RESIDUAL, par, d, "K"), K[par], atol=1e-14)
        np.testing.assert_allclose(O.reconstruct_layer(unit, O.RESIDUAL, par, d, "V"), V[par], atol=1e-14)


def test_exact_mode_keeps_inputs_bitwise():
    rng = np.random.default_rng(6)
    K = gen.round_bf16_f32(rng.standard_normal((2, 5, 8)).astype(np.float32))
    unit = O.compress_unit(K, K, O.EXACT, 3, "bf16")
    np.testing.assert_array_equal(unit["K0"], K[0])
    np.testing.assert_array_equal(unit["K1"], K[1])


def test_needle_recovery_tiny():
    """The planted needle channels are exactly the top-k residual at needle tokens."""
    w = WORKLOADS["tiny"]
    for h in range(w.n_kv_heads):
        K, V, info = gen.segment(w, 0, 0, h)
        idxK = O.residual_channels(K[0], K[1], w.topk)
        idxV = O.residual_channels(V[0], V[1], w.topk)
        for pos, layer, ch in info["needles"]:
            assert layer == 1
            assert idxK[pos].tolist() == ch.tolist()
            assert idxV[pos].tolist() == ch.tolist()


# ---------------------------------------------------------------- hand-worked example
def test_golden_worked_example():
    g = _golden()
    K = np.stack([g["K0"].reshape(2, 4), g["K1"].reshape(2, 4)])
    V = np.stack([g["V0"].reshape(2, 4), g["V1"].reshape(2, 4)])
    unit = O.compress_unit(K, V, O.RESIDUAL, 1, "f32")
    np.testing.assert_array_equal(unit["MK"].reshape(-1), g["MK"])
    np.testing.assert_array_equal(unit["MV"].reshape(-1), g["MV"])
    np.testing.assert_array_equal(unit["IK"].reshape(-1), g["IK"])
    np.testing.assert_array_equal(unit["VK"].reshape(-1), g["VK"])
    np.testing.assert_array_equal(unit["IV"].reshape(-1), g["IV"])
    np.testing.assert_array_equal(unit["VV"].reshape(-1), g["VV"])
    q = np.array([[0.0, 0.0, 0.0, math.log(3.0) / 2.0]])
    out = O.decode_unit(unit, O.RESIDUAL, 0, q, 0.5, 4)
    np.testing.assert_allclose(out[0], g["OUT_R_L0"], atol=1e-14)
    # shared mode, layer 1
    sunit = O.compress_unit(K, V, O.SHARED, 1, "f32")
    out = O.decode_unit(sunit, O.SHARED, 1, q, 0.5, 4)
    s3 = 3.0 * math.sqrt(3.0)
    np.testing.assert_allclose(out[0], (s3 * np.array([1, 0, 1, 0]) + np.array([0, 2, 0, 3])) / (s3 + 1), atol=1e-14)
    # routing loss
    Q2 = np.zeros((2, 1, 1, 4))
    Q2[:, 0, 0, 3] = 2.0
    np.testing.assert_allclose(O.routing_errors(K, Q2, 1), g["E"], atol=1e-13)
    om = O.omega(4, 1, "f32")
    np.testing.assert_array_equal(om, g["OMEGA"])
    E = g["E"][None]
    got = [int(O.route(E, om, lam)[0]) for lam in (1.0, 4.0, 100.0)]
    assert got == g["ROUTE_L1_L4_L100"].astype(int).tolist()


# ---------------------------------------------------------------- decode
def _textbook_attention(q, K, V, scale):
    return scipy.special.softmax((q @ K.T) * scale, axis=-1) @ V


def test_exact_heads_equal_textbook_attention():
    rng = np.random.default_rng(7)
    K = rng.standard_normal((2, 40, 8))
    V = rng.standard_normal((2, 40, 8))
    unit = O.compress_unit(K, V, O.EXACT, 3, "f64")
    q = rng.standard_normal((3, 8))
    for layer in (0, 1):
        np.testing.assert_allclose(O.decode_unit(unit, O.EXACT, layer, q, 0.3, 8),
                                   _textbook_attention(q, K[layer], V[layer], 0.3), rtol=1e-13, atol=1e-14)


def test_tiny_brute_force_softmax():
    rng = np.random.default_rng(8)
    T, d = 5, 3
    K = rng.standard_normal((T, d))
    V = rng.standard_normal((T, d))
    q = rng.standard_normal(d)
    w = [math.exp(sum(q[c] * K[t][c] for c in range(d)) * 0.7) for t in range(T)]
    ref = [sum(w[t] * V[t][c] for t in range(T)) / sum(w) for c in range(d)]
    np.testing.assert_allclose(O.attention(q[None], K, V, 0.7)[0], ref, rtol=1e-13)


def test_single_token_and_zero_query():
    rng = np.random.default_rng(9)
    K = rng.standard_normal((2, 1, 8))
    V = rng.standard_normal((2, 1, 8))
    for mode in O.MODES:
        unit = O.compress_unit(K, V, mode, 2, "f64")
        out = O.decode_unit(unit, mode, 1, rng.standard_normal((2, 8)), 1.0, 8)
        np.testing.assert_allclose(out, np.repeat(O.reconstruct_layer(unit, mode, 1, 8, "V"), 2, 0), atol=1e-14)
    K = rng.standard_normal((2, 17, 8))
    V = rng.standard_normal((2, 17, 8))
    for mode in O.MODES:
        unit = O.compress_unit(K, V, mode, 2, "f64")
        out = O.decode_unit(unit, mode, 0, np.zeros((1, 8)), 1.0, 8)
        np.testing.assert_allclose(out[0], O.reconstruct_layer(unit, mode, 0, 8, "V").mean(0), atol=1e-14)


def test_shared_heads_same_output_in_both_layers():
    rng = np.random.default_rng(10)
    K = rng.standard_normal((2, 30, 8))
    V = rng.standard_normal((2, 30, 8))
    unit = O.compress_unit(K, V, O.SHARED, 2, "f32")
    q = rng.standard_normal((2, 8))
    np.testing.assert_array_equal(O.decode_unit(unit, O.SHARED, 0, q, 0.4, 8),
                                  O.decode_unit(unit, O.SHARED, 1, q, 0.4, 8))


def test_shared_mode_is_pair_mean_and_residual_adds_signed_half_difference():
    rng = np.random.default_rng(11)
    K = rng.standard_normal((2, 6, 8))
    unit = O.compress_unit(K, K, O.RESIDUAL, 8, "f64")
    np.testing.assert_allclose(unit["MK"], (K[0] + K[1]) / 2, atol=1e-15)
    np.testing.assert_allclose(unit["VK"], (K[0] - K[1]) / 2, atol=1e-15)


# ---------------------------------------------------------------- Eq. (2)
def _brute_routing(K2, Q2, k):
    """Eq. (2) with explicit loops over layers, heads, probe rows and tokens."""
    _, T, d = K2.shape
    nl, G, P, _ = Q2.shape
    idx = O.residual_channels(K2[0], K2[1], k)
    res = []
    for mode in O.MODES:
        tot = 0.0
        for l in range(nl):
            sign = 1.0 if l == 0 else -1.0
            for g in range(G):
                for p in range(P):
                    for t in range(T):
                        # K^(m) - K for layer l, written out per channel
                        s = 0.0
                        for c in range(d):
                            half = (K2[0, t, c] - K2[1, t, c]) / 2.0
                            if mode == O.EXACT:
                                diff = 0.0
                            elif mode == O.SHARED or c not in idx[t]:
                                diff = -sign * half
                            else:
                                diff = 0.0
                            s += Q2[l, g, p, c] * diff
                        tot += (s / math.sqrt(d)) ** 2
        res.append(tot / (nl * G * P))
    return np.array(res)


def test_routing_errors_brute_force():
    rng = np.random.default_rng(12)
    K2 = rng.standard_normal((2, 6, 5)).astype(np.float32).astype(np.float64)
    Q2 = rng.standard_normal((2, 2, 3, 5))
    np.testing.assert_allclose(O.routing_errors(K2, Q2, 2), _brute_routing(K2, Q2, 2), rtol=1e-12, atol=1e-15)


def test_routing_errors_invariants():
    rng = np.random.default_rng(13)
    K2 = rng.standard_normal((2, 20, 8))
    Q2 = rng.standard_normal((2, 2, 4, 8))
    E = O.routing_errors(K2, Q2, 3)
    assert E[O.EXACT] == 0.0
    assert E[O.RESIDUAL] <= E[O.SHARED]
    assert O.routing_errors(K2, Q2, 8)[O.RESIDUAL] < 1e-25           # k = d
    same = np.stack([K2[0], K2[0]])
    Es = O.routing_errors(same, Q2, 3)
    # identical layers: zero up to the fp64 noise of reconstructing K through F^T F
    assert Es[O.SHARED] < 1e-28 and Es[O.RESIDUAL] < 1e-28
    om = O.omega(8, 3, "bf16")
    for lam in (1e-20, 1e-3, 1.0, 1e6):
        assert int(O.route(Es[None], om, lam)[0]) == O.SHARED
    # with exactly zero errors the tie at lambda = 0 goes to the cheapest mode
    assert int(O.route(np.zeros((1, 3)), om, 0.0)[0]) == O.SHARED


def test_routing_error_statistics():
    """E_S is about T (1 - rho) / (2 d) for q ~ N(0, I/d)."""
    rng = np.random.default_rng(14)
    T, d, rho = 4096, 32, 0.8
    x0 = rng.standard_normal((T, d))
    x1 = rho * x0 + math.sqrt(1 - rho * rho) * rng.standard_normal((T, d))
    Q2 = rng.standard_normal((2, 2, 64, d)) / math.sqrt(d)
    E = O.routing_errors(np.stack([x0, x1]), Q2, 4)
    assert abs(E[O.SHARED] / (T * (1 - rho) / (2 * d)) - 1.0) < 0.08


# ---------------------------------------------------------------- routing and bytes
def test_omega_closed_form():
    np.testing.assert_allclose(O.omega(128, 16, "bf16"), [0.5, 0.59375, 1.0])
    np.testing.assert_allclose(O.omega(64, 8, "f32"), [0.5, 0.578125, 1.0])


def test_cache_bytes_tiny_by_hand():
    w = WORKLOADS["tiny"]
    modes = gen.fixed_modes(w)[None]
    # T*d*e = 512*64*4 = 131072 per dense plane; residual planes 512*8 = 4096 (u8)
    # and 512*8*4 = 16384 (fp32); S = 2 planes, R = 2 + 4 small, E = 4 planes.
    assert O.cache_bytes(w.seq_lens, modes, 64, 8, "f32") == 1392640


def test_plane_padding():
    assert O.unit_bytes(O.SHARED, 1, 64, 8, "bf16") == 2 * 256
    assert O.unit_bytes(O.RESIDUAL, 3, 64, 8, "bf16") == 2 * 512 + 2 * (256 + 256)
    assert O.unit_bytes(O.EXACT, 2, 128, 16, "bf16") == 4 * 512


def test_route_limits():
    rng = np.random.default_rng(15)
    E = np.abs(rng.standard_normal((50, 3)))
    E[:, 1] = E[:, 0] * 0.5
    E[:, 2] = 0.0
    om = O.omega(128, 16, "bf16")
    assert (O.route(E, om, 0.0) == O.EXACT).all()
    assert (O.route(E, om, math.inf) == O.SHARED).all()
    assert (O.route(E, om, 1e30) == O.SHARED).all()


def test_route_breakpoint_ties_go_to_the_cheaper_mode():
    """At lambda equal to a unit's breakpoint its two modes cost the same, and the
    tie rule gives the cheaper one, even where E_a + lam O_a and E_b + lam O_b
    evaluated in floating point round apart (cases searched for below)."""
    rng = np.random.default_rng(151)
    om = O.omega(128, 16, "bf16")
    rounded_apart = 0
    for _ in range(4000):
        E = np.array([rng.uniform(1, 100), 0.0, 0.0])
        E[1] = E[0] * rng.uniform(0.2, 0.8)
        for a, b in ((0, 1), (1, 2), (0, 2)):
            lam = (E[a] - E[b]) / (om[b] - om[a])
            if not lam > 0:
                continue
            ca, cb = E[a] + lam * om[a], E[b] + lam * om[b]
            rounded_apart += ca != cb
            # with only modes a and b competing (the third priced out), the tie goes to a
            E2 = E.copy()
            third = 3 - a - b
            E2[third] = 1e300
            assert int(O.route(E2[None], om, lam)[0]) == a, (E, a, b, lam)
            # a hair below the breakpoint the costlier, more accurate mode wins
            assert int(O.route(E2[None], om, np.nextafter(lam, 0.0))[0]) == b
    assert rounded_apart > 0          # the floating-point costs do break some of these ties


def test_route_budget_minimal_lambda_brute_force():
    rng = np.random.default_rng(16)
    T, d, k = 1000, 64, 8
    for trial in range(5):
        E = np.abs(rng.standard_normal((12, 3))) * 10
        E[:, 1] = E[:, 0] * rng.uniform(0.2, 0.9, 12)
        E[:, 2] = 0.0
        om = O.omega(d, k, "bf16")
        seg = {m: O.unit_bytes(m, T, d, k, "bf16") for m in O.MODES}

        def fp(lam):
            return sum(seg[int(m)] for m in O.route(E, om, lam))

        lo, hi = fp(math.inf), fp(0.0)
        budget = int(lo + (hi - lo) * rng.uniform(0.1, 0.9))
        modes, lam, ok = O.route_budget(E, T, d, k, "bf16", budget)
        assert ok and fp(lam) <= budget
        grid = np.linspace(0, lam, 2000, endpoint=False)
        assert all(fp(x) > budget for x in grid)
        # footprint never grows with lambda
        lams = np.linspace(0, 3 * lam + 1, 500)
        fps = [fp(x) for x in lams]
        assert all(a >= b for a, b in zip(fps, fps[1:]))
    modes, lam, ok = O.route_budget(E, T, d, k, "bf16", 10)
    assert not ok and (modes == O.SHARED).all()


def test_gqa_is_per_query_head_attention():
    rng = np.random.default_rng(17)
    K = rng.standard_normal((2, 25, 8))
    V = rng.standard_normal((2, 25, 8))
    unit = O.compress_unit(K, V, O.RESIDUAL, 3, "f32")
    q = rng.standard_normal((4, 8))
    full = O.decode_unit(unit, O.RESIDUAL, 1, q, 0.35, 8)
    for g in range(4):
        np.testing.assert_allclose(full[g], O.decode_unit(unit, O.RESIDUAL, 1, q[g:g + 1], 0.35, 8)[0], rtol=1e-14)


# ---------------------------------------------------------------------------
# OCP FP8 E4M3 coefficient storage (cache type bf16_e4m3)
# ---------------------------------------------------------------------------
def _e4m3_grid():
    """Every finite E4M3 value, enumerated from the format: sign, exponent
    field 0..15 (bias 7, field 0 subnormal), mantissa 0..7, minus S.1111.111."""
    vals = []
    for e in range(16):
        for m in range(8):
            if e == 15 and m == 7:
                continue
            v = m * 2.0 ** -9 if e == 0 else (1 + m / 8) * 2.0 ** (e - 7)
            vals.append((v, m))
    return vals


def _nearest_e4m3(x):
    """Brute force: the grid value nearest to x; at an exact midpoint the one
    with an even mantissa field; beyond 448 saturate."""
    grid = _e4m3_grid()
    a = abs(x)
    if a >= 448:
        return math.copysign(448.0, x)
    best = min(grid, key=lambda vm: (abs(vm[0] - a), vm[1] & 1))
    return math.copysign(best[0], x)


def test_e4m3_grid_is_fixed():
    grid = np.array([v for v, _ in _e4m3_grid()])
    assert len(grid) == 127 and grid.max() == 448.0 and grid[1] == 2.0 ** -9
    np.testing.assert_array_equal(O.round_e4m3(grid), grid)
    np.testing.assert_array_equal(O.round_e4m3(-grid), -grid)


def test_e4m3_rounding_matches_brute_force():
    rng = np.random.default_rng(71)
    grid = sorted(v for v, _ in _e4m3_grid())
    mids = [(a + b) / 2 for a, b in zip(grid[:-1], grid[1:])]           # exact ties
    xs = np.concatenate([rng.standard_normal(3000) * 3, rng.uniform(-500, 500, 1000),
                         rng.uniform(-0.02, 0.02, 1000), mids, [-m for m in mids],
                         [449.0, 464.0, 470.0, 479.9, 480.0, 1e6, -1e6, 2.0 ** -10, 3 * 2.0 ** -10, 0.0]])
    want = np.array([_nearest_e4m3(float(x)) for x in xs])
    np.testing.assert_array_equal(O.round_e4m3(xs), want)


def test_e4m3_cache_bytes_closed_form():
    # coefficient planes one byte per element, exact heads bf16, indices uint8
    T, d, k = 1000, 128, 16
    pad = lambda n: -(-n // 256) * 256
    assert O.unit_bytes(O.SHARED, T, d, k, "bf16_e4m3") == 2 * pad(T * d)
    assert O.unit_bytes(O.RESIDUAL, T, d, k, "bf16_e4m3") == 2 * pad(T * d) + 2 * (pad(T * k) + pad(T * k))
    assert O.unit_bytes(O.EXACT, T, d, k, "bf16_e4m3") == 4 * pad(T * d * 2)
    np.testing.assert_allclose(O.omega(d, k, "bf16_e4m3"), [256 / 1024, (256 + 64) / 1024, 1.0])
    # FP8 shared planes fill whole 1 KB blocks (1001 rows of 64 channels: 62.56 blocks -> 63)
    assert O.unit_bytes(O.SHARED, 1001, 64, 8, "bf16_e4m3") == 2 * 63 * 1024
    assert O.unit_bytes(O.RESIDUAL, 1001, 64, 8, "bf16_e4m3") == 2 * 63 * 1024 + 2 * (pad(1001 * 8) + pad(1001 * 8))
    assert O.unit_bytes(O.SHARED, 1001, 64, 8, "bf16") == 2 * pad(1001 * 64 * 2)


def test_e4m3_unit_stores_rounded_coefficients():
    rng = np.random.default_rng(5)
    K2 = O.round_bf16(rng.standard_normal((2, 40, 64)))
    V2 = O.round_bf16(rng.standard_normal((2, 40, 64)))
    u = O.compress_unit(K2, V2, O.RESIDUAL, 8, "bf16_e4m3")
    ub = O.compress_unit(K2, V2, O.RESIDUAL, 8, "bf16")
    # same channels; values are the E4M3 rounding of the exact mean / half difference
    np.testing.assert_array_equal(u["IK"], ub["IK"])
    np.testing.assert_array_equal(u["MK"], O.round_e4m3((K2[0] + K2[1]) / 2))
    D = (V2[0] - V2[1]) / 2
    np.testing.assert_array_equal(u["VV"], O.round_e4m3(np.take_along_axis(D, u["IV"], axis=-1)))
    e = O.compress_unit(K2, V2, O.EXACT, 8, "bf16_e4m3")
    np.testing.assert_array_equal(e["K1"], K2[1])                   # exact heads keep bf16


# ---------------------------------------------------------------- B = 4 blocks and the mixed schedule
def test_block_schedules():
    # Section 4: blocks of four by default, pairs for the first and the last four layers
    assert [B for _, B in O.block_schedule(32, O.MIXED)] == [2, 2, 4, 4, 4, 4, 4, 4, 2, 2]
    for L, sched in [(32, O.MIXED), (8, O.MIXED), (12, O.MIXED), (16, O.QUADS), (6, O.PAIRS)]:
        blocks = O.block_schedule(L, sched)
        assert [l for f, B in blocks for l in range(f, f + B)] == list(range(L))
        assert all(f % B == 0 for f, B in blocks)
    assert all(B == 2 for f, B in O.block_schedule(40, O.MIXED) if f < 4 or f >= 36)
    assert all(B == 4 for f, B in O.block_schedule(40, O.MIXED) if 4 <= f < 36)
    for bad in [(10, O.MIXED), (6, O.MIXED), (6, O.QUADS), (7, O.PAIRS)]:
        with pytest.raises(ValueError):
            O.block_schedule(*bad)
    assert O.block_of_layer(32, O.MIXED, 5) == (2, 4, 1)
    assert O.block_of_layer(32, O.MIXED, 29) == (8, 2, 1)
    assert O.block_of_layer(12, O.QUADS, 11) == (2, 4, 3)


def test_dct4_keys_are_coefficient_magnitudes():
    # the keys are |Z_j| of scipy's orthonormal DCT-II along the layer axis, to float64 rounding
    rng = np.random.default_rng(21)
    X = O.round_bf16(rng.standard_normal((4, 50, 16)) * 3.0)
    key = O.residual_keys_dct4(X)
    assert key.dtype == np.float64 and key.shape == (50, 16, 3)
    ref = np.abs(np.moveaxis(scipy.fft.dct(X, type=2, norm="ortho", axis=0)[1:], 0, -1))
    bound = 1e-14 * np.abs(X).max(axis=0)[..., None]
    assert np.all(np.abs(key - ref) <= bound)


def test_dct4_codes_brute_force():
    rng = np.random.default_rng(22)
    for trial in range(40):
        d = int(rng.integers(1, 4))
        # small integers force ties (zeros, equal second differences)
        X = rng.integers(-2, 3, size=(4, 1, d)).astype(np.float32)
        key = O.residual_keys_dct4(X)[0]                       # [d][3]
        flat = [float(key[c, j]) for c in range(d) for j in range(3)]
        code_of = [4 * c + j + 1 for c in range(d) for j in range(3)]
        for k in range(0, 3 * d + 1):
            got = O.residual_codes_dct4(X, k)[0].tolist()
            want = [code_of[i] for i in _brute_topk(flat, k)] if k else []
            assert got == want, (X.ravel(), k)


def test_dct4_parseval_block_error():
    # the reconstruction error over the block is the energy of the dropped coefficients
    rng = np.random.default_rng(23)
    T, d = 30, 8
    X = rng.standard_normal((4, T, d)).astype(np.float32).astype(np.float64)
    Z = scipy.fft.dct(X, type=2, norm="ortho", axis=0)
    t = np.arange(T)[:, None]
    for k in (0, 1, 5, 13, 23):
        codes = O.residual_codes_dct4(X, k)
        kept = np.zeros(Z.shape, dtype=bool)
        kept[0] = True
        kept[codes & 3, t, codes >> 2] = True
        dropped = np.sum(np.where(kept, 0.0, Z) ** 2, axis=(0, 2))
        Kr = O.candidate_keys(X, O.RESIDUAL, k)
        np.testing.assert_allclose(np.sum((Kr - X) ** 2, axis=(0, 2)), dropped, rtol=1e-10, atol=1e-12)
        # greedy by magnitude: no dropped coefficient is larger than a kept one
        if 0 < k < 3 * d:
            hf = np.abs(Z[1:])
            kk = kept[1:]
            assert np.all(np.max(np.where(kk, 0.0, hf), axis=(0, 2)) <=
                          np.min(np.where(kk, hf, np.inf), axis=(0, 2)) + 1e-6)
    np.testing.assert_allclose(O.candidate_keys(X, O.RESIDUAL, 3 * d), X, atol=1e-12)   # k = 3d
    np.testing.assert_allclose(O.candidate_keys(X, O.SHARED, 0), np.broadcast_to(X.mean(0), X.shape), atol=1e-14)


def test_dct4_identical_layers():
    rng = np.random.default_rng(24)
    X = rng.standard_normal((9, 16)).astype(np.float32)
    X4 = np.stack([X] * 4)
    unit = O.compress_unit(X4, X4, O.RESIDUAL, 5, "f32")
    np.testing.assert_array_equal(unit["IK"], np.tile([1, 2, 3, 5, 6], (9, 1)))
    np.testing.assert_array_equal(unit["VK"], 0.0)
    np.testing.assert_array_equal(unit["MK"], X.astype(np.float64))
    Q = rng.standard_normal((4, 2, 3, 16))
    E = O.routing_errors(X4.astype(np.float64), Q, 5)
    assert E[O.SHARED] < 1e-26 and E[O.RESIDUAL] < 1e-26 and E[O.EXACT] == 0.0


def _idct_rebuild(unit, which, T, d):
    """K~ of all four layers: Z from the stored planes, then scipy's inverse DCT-II."""
    Z = np.zeros((4, T, d))
    Z[0] = 2.0 * unit["M" + which]                 # the stored plane is Z_0 / 2 (the layer mean)
    for t in range(T):
        for code, v in zip(unit["I" + which][t], unit["V" + which][t]):
            Z[code & 3, t, code >> 2] = v
    return scipy.fft.idct(Z, type=2, norm="ortho", axis=0)


def test_dct4_decode_brute_force():
    rng = np.random.default_rng(25)
    T, d, G = 6, 4, 2
    K = rng.standard_normal((4, T, d))
    V = rng.standard_normal((4, T, d))
    for mode in (O.SHARED, O.RESIDUAL, O.EXACT):
        unit = O.compress_unit(K, V, mode, 3, "f64")
        if mode == O.EXACT:
            Kt, Vt = K, V
        elif mode == O.SHARED:
            Kt = np.broadcast_to(K.mean(0), K.shape)
            Vt = np.broadcast_to(V.mean(0), V.shape)
        else:
            Kt, Vt = _idct_rebuild(unit, "K", T, d), _idct_rebuild(unit, "V", T, d)
        for p in range(4):
            q = rng.standard_normal((G, d))
            want = np.zeros((G, d))
            for g in range(G):
                s = [sum(q[g, c] * Kt[p, t, c] for c in range(d)) * 0.4 for t in range(T)]
                w = [math.exp(x - max(s)) for x in s]
                for t in range(T):
                    want[g] += w[t] / sum(w) * Vt[p, t]
            got = O.decode_unit(unit, mode, 8 + p, q, 0.4, d, B=4)
            np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)


def test_dct4_unit_stores_codes_and_coefficients():
    rng = np.random.default_rng(26)
    X = O.round_bf16(rng.standard_normal((4, 7, 8)))
    unit = O.compress_unit(X, X, O.RESIDUAL, 6, "bf16")
    Z = scipy.fft.dct(X, type=2, norm="ortho", axis=0)
    codes = unit["IK"]
    assert codes.shape == (7, 6) and np.all(np.diff(codes, axis=-1) > 0)
    assert np.all((codes & 3) >= 1) and np.all((codes >> 2) < 8)
    t = np.arange(7)[:, None]
    z = Z[codes & 3, t, codes >> 2]
    # nearest bf16 (within half a unit in the last place; scipy's rounding noise decides exact ties)
    np.testing.assert_array_equal(unit["VK"], O.round_bf16(unit["VK"]))
    assert np.all(np.abs(unit["VK"] - z) <= 2.0 ** -8 * np.abs(z) * (1 + 1e-12))
    np.testing.assert_array_equal(unit["MK"], O.round_bf16(X.mean(0)))


def _brute_routing4(K4, Q4, k):
    """Eq. (2) for a block of four with explicit loops; K^ rebuilt by scipy's inverse DCT."""
    _, T, d = K4.shape
    _, G, P, _ = Q4.shape
    Z = scipy.fft.dct(K4, type=2, norm="ortho", axis=0)
    codes = O.residual_codes_dct4(K4, k)
    res = []
    for mode in O.MODES:
        Zm = np.zeros_like(Z)
        if mode == O.EXACT:
            Zm = Z.copy()
        else:
            Zm[0] = Z[0]
            if mode == O.RESIDUAL:
                for t in range(T):
                    for code in codes[t]:
                        Zm[code & 3, t, code >> 2] = Z[code & 3, t, code >> 2]
        Kh = scipy.fft.idct(Zm, type=2, norm="ortho", axis=0)
        tot = 0.0
        for l in range(4):
            for g in range(G):
                for p in range(P):
                    for t in range(T):
                        s = sum(Q4[l, g, p, c] * (Kh[l, t, c] - K4[l, t, c]) for c in range(d))
                        tot += (s / math.sqrt(d)) ** 2
        res.append(tot / (4 * G * P))
    return np.array(res)


def test_dct4_routing_errors_brute_force():
    rng = np.random.default_rng(27)
    K4 = rng.standard_normal((4, 5, 4)).astype(np.float32).astype(np.float64)
    Q4 = rng.standard_normal((4, 2, 3, 4))
    got = O.routing_errors(K4, Q4, 3)
    want = _brute_routing4(K4, Q4, 3)
    np.testing.assert_allclose(got[:2], want[:2], rtol=1e-11)
    assert got[O.EXACT] == 0.0 and abs(want[O.EXACT]) < 1e-25


def test_dct4_bytes_closed_form():
    # B = 4: 16-bit codes; exact heads keep all four layers
    np.testing.assert_allclose(O.omega(128, 16, "bf16", 4), [0.25, 0.3125, 1.0])
    np.testing.assert_allclose(O.omega(64, 8, "bf16_e4m3", 4), [0.125, 0.171875, 1.0])
    assert O.unit_bytes(O.RESIDUAL, 3, 64, 8, "bf16", 4) == 2 * 512 + 2 * (256 + 256)
    assert O.unit_bytes(O.RESIDUAL, 100, 64, 8, "bf16", 4) == 2 * 12800 + 2 * (1792 + 1792)
    assert O.unit_bytes(O.EXACT, 2, 128, 16, "bf16", 4) == 8 * 512
    # 12 layers mixed = pairs (0,1), (2,3), quad (4..7), pairs (8,9), (10,11); 1 KV head, T = 256
    modes = np.array([[[O.SHARED], [O.RESIDUAL], [O.EXACT], [O.RESIDUAL], [O.SHARED]]])
    sizes = [B for _, B in O.block_schedule(12, O.MIXED)]
    # bf16, d = 64: coefficient plane 32768 B; index planes 256*8 (B = 2) or 256*16 (B = 4)
    s = 2 * 32768
    r2 = s + 2 * (2048 + 4096)
    e4 = 8 * 32768
    assert O.cache_bytes([256], modes, 64, 8, "bf16", sizes) == s + r2 + e4 + r2 + s


def test_route_budget_mixed_sizes_brute_force():
    rng = np.random.default_rng(28)
    T, d, k = 1000, 64, 8
    sizes = [2, 2, 4, 4, 2, 2] * 2
    for trial in range(5):
        E = np.abs(rng.standard_normal((12, 3))) * 10
        E[:, 1] = E[:, 0] * rng.uniform(0.2, 0.9, 12)
        E[:, 2] = 0.0
        om = np.stack([O.omega(d, k, "bf16", B) for B in sizes])

        def fp(lam):
            return sum(O.unit_bytes(int(m), T, d, k, "bf16", B) for m, B in zip(O.route(E, om, lam), sizes))

        lo, hi = fp(math.inf), fp(0.0)
        budget = int(lo + (hi - lo) * rng.uniform(0.1, 0.9))
        modes, lam, ok = O.route_budget(E, T, d, k, "bf16", budget, sizes)
        assert ok and fp(lam) <= budget
        assert all(fp(x) > budget for x in np.linspace(0, lam, 2000, endpoint=False))


# ---------------------------------------------------------------- generation: spans and the exact tail
@pytest.mark.parametrize("B", [2, 4])
def test_spans_are_token_local(B):
    """Compressing a sequence in pieces gives the same cache as compressing it whole
    (every per-token quantity is token-local), so decode over the spans is decode
    over the whole."""
    rng = np.random.default_rng(40 + B)
    T, d = 37, 16
    K = O.round_bf16(rng.standard_normal((B, T, d)))
    V = O.round_bf16(rng.standard_normal((B, T, d)))
    for mode in O.MODES:
        whole = O.compress_unit(K, V, mode, 5, "bf16")
        cut = [0, 11, 12, 30, T]
        spans = [(O.compress_unit(K[:, a:b], V[:, a:b], mode, 5, "bf16"), mode, B) for a, b in zip(cut, cut[1:])]
        for layer in range(B):
            q = rng.standard_normal((3, d))
            want = O.decode_unit(whole, mode, layer, q, 0.25, d, B)
            got = O.decode_spans(spans, np.zeros((0, d)), np.zeros((0, d)), layer, q, 0.25, d)
            np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)


def test_tail_is_exact_attention():
    rng = np.random.default_rng(44)
    T, n, d = 20, 7, 8
    K = rng.standard_normal((2, T, d))
    V = rng.standard_normal((2, T, d))
    tk, tv = rng.standard_normal((n, d)), rng.standard_normal((n, d))
    q = rng.standard_normal((2, d))
    unit = O.compress_unit(K, V, O.EXACT, 3, "f64")
    for layer in (0, 1):
        got = O.decode_spans([(unit, O.EXACT, 2)], tk, tv, layer, q, 0.3, d)
        Kc, Vc = np.concatenate([K[layer], tk]), np.concatenate([V[layer], tv])
        want = scipy.special.softmax(q @ Kc.T * 0.3, axis=-1) @ Vc
        np.testing.assert_allclose(got, want, rtol=1e-12)
    only_tail = O.decode_spans([], tk, tv, 0, q, 0.3, d)
    np.testing.assert_allclose(only_tail, scipy.special.softmax(q @ tk.T * 0.3, axis=-1) @ tv, rtol=1e-12)
    assert np.all(O.decode_spans([], np.zeros((0, d)), np.zeros((0, d)), 0, q, 0.3, d) == 0.0)


def test_refresh_routes_a_hand_worked_span():
    """One token, d = 4, k = 1, a probe row of ones in both layers: x0 = (2, 1, 0, 0),
    x1 = 0.  D = (1, 1/2, 0, 0); the shared reconstruction misses -+D, so each
    layer's logit error is (1 + 1/2) / sqrt(4) = 3/4 and E_S = 9/16; the residual
    keeps channel 0 and misses -+(0, 1/2, 0, 0): E_R = (1/4)^2 = 1/16.  bf16,
    d = 4, k = 1: Omega = (16, 16 + 2 (1 + 2), 32) / 32 = (1/2, 11/16, 1).
    Breakpoints: R|E at (1/16) / (5/16) = 1/5, S|R at (1/2) / (3/16) = 8/3, so
    exact below 1/5, residual up to 8/3, shared above (ties to the cheaper)."""
    K = np.zeros((2, 1, 4))
    K[0, 0] = [2.0, 1.0, 0.0, 0.0]
    Q = np.ones((2, 1, 1, 4))
    np.testing.assert_allclose(O.routing_errors(K, Q, 1), [9 / 16, 1 / 16, 0.0], rtol=0, atol=1e-15)
    np.testing.assert_array_equal(O.omega(4, 1, "bf16"), [0.5, 11 / 16, 1.0])
    om = O.omega(4, 1, "bf16")
    lam_re = (1 / 16 - 0.0) / (om[2] - om[1])
    lam_sr = (9 / 16 - 1 / 16) / (om[1] - om[0])
    want = [(0.0, O.EXACT), (0.1, O.EXACT), (lam_re, O.RESIDUAL), (1.0, O.RESIDUAL), (2.5, O.RESIDUAL),
            (lam_sr, O.SHARED), (3.0, O.SHARED), (math.inf, O.SHARED)]
    for lam, m in want:
        assert O.refresh_modes(K, Q, 1, "bf16", lam) == m, (lam, m)
    # a block of four with the same deviations in its four layers' halves routes by Omega of B = 4
    om4 = O.omega(4, 1, "bf16", 4)
    np.testing.assert_array_equal(om4, [16 / 64, (16 + 2 * (2 + 2)) / 64, 1.0])


def test_refresh_routes_the_span():
    rng = np.random.default_rng(45)
    X = rng.standard_normal((9, 16))
    same = np.stack([X, X])
    Q = rng.standard_normal((2, 2, 5, 16))
    # identical layers: E_S is zero up to the fp64 noise of F^T F, so any positive penalty picks shared
    assert O.refresh_modes(same, Q, 4, "bf16", 1e-20) == O.SHARED
    far = np.stack([X, -X])
    assert O.refresh_modes(far, Q, 4, "bf16", 0.0) == O.EXACT             # lambda 0: zero error wins
    assert O.refresh_modes(far, Q, 4, "bf16", math.inf) == O.SHARED


# ---------------------------------------------------------------- token-level residual set
@pytest.mark.parametrize("B", [2, 4])
def test_token_score_is_the_shared_logit_change(B):
    """s_t = max over probe rows of |q . (K_t - K^S_t)| (the paper's score); e_t sums the
    squares, so sum_t e_t / (B G P d) is E_S."""
    rng = np.random.default_rng(50 + B)
    T, d, G, P = 40, 16, 2, 3
    K = O.round_bf16(rng.standard_normal((B, T, d)))
    Q = O.round_bf16(rng.standard_normal((B, G, P, d)))
    s, e = O.token_scores(K, Q)
    Ks = O.candidate_keys(K, O.SHARED, 0)
    brute_s = np.zeros(T)
    brute_e = np.zeros(T)
    for l in range(B):
        for g in range(G):
            for p in range(P):
                for t in range(T):
                    v = sum(Q[l, g, p, c] * (K[l, t, c] - Ks[l, t, c]) for c in range(d))
                    brute_s[t] = max(brute_s[t], abs(v))
                    brute_e[t] += v * v
    np.testing.assert_allclose(s, brute_s, rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(e, brute_e, rtol=1e-12, atol=1e-12)
    E = O.routing_errors(K, Q, 0)
    np.testing.assert_allclose(e.sum() / (B * G * P * d), E[O.SHARED], rtol=1e-12)


def test_token_deviations_are_exact_differences():
    # pairs: x0 - M = (x0 - x1) / 2 and its negation; fours: x_l minus the four-layer mean, exactly
    x = np.array([[1.0, 3.0], [1.0 + 2 ** -7, -5.0]])[:, None, :]     # [2][1][2]
    dev = O.token_deviations(x)
    assert dev[0, 0, 0] == -2 ** -8 and dev[1, 0, 0] == 2 ** -8 and dev[0, 0, 1] == 4.0 and dev[1, 0, 1] == -4.0
    X4 = np.array([1.0, 2.0, 4.0, 1.0 + 2 ** -20])[:, None, None]
    M = (8.0 + 2 ** -20) / 4
    np.testing.assert_array_equal(O.token_deviations(X4)[:, 0, 0], X4[:, 0, 0] - M)


def test_residual_tokens_brute_force():
    rng = np.random.default_rng(53)
    for trial in range(30):
        T = int(rng.integers(1, 9))
        s = rng.integers(0, 3, size=T).astype(np.float64)
        for n in range(T + 1):
            got = O.residual_tokens(s, n).tolist()
            assert got == (_brute_topk(s.tolist(), n) if n else [])
    assert O.n_residual_tokens(32768, 50000) == 1639 and O.n_residual_tokens(100, 0) == 0
    assert O.n_residual_tokens(3, 1) == 1 and O.n_residual_tokens(1000000, 1) == 1


@pytest.mark.parametrize("B", [2, 4])
def test_token_routing_errors_limits_and_split(B):
    rng = np.random.default_rng(54 + B)
    T, d, G, P = 60, 8, 2, 4
    K = O.round_bf16(rng.standard_normal((B, T, d)))
    Q = rng.standard_normal((B, G, P, d))
    E0 = O.routing_errors_tokens(K, Q, 0)
    Eall = O.routing_errors_tokens(K, Q, 1000000)
    Ech = O.routing_errors(K, Q, 0)
    assert Eall[O.RESIDUAL] < 1e-25 and E0[O.EXACT] == 0.0
    np.testing.assert_allclose(E0[O.RESIDUAL], Ech[O.SHARED], rtol=1e-12)
    np.testing.assert_allclose(E0[O.SHARED], Ech[O.SHARED], rtol=1e-12)
    # E_R = E_S minus the kept tokens' own contributions (Eq. 2 splits over tokens)
    ppm = 150000
    E = O.routing_errors_tokens(K, Q, ppm)
    s, _ = O.token_scores(K, Q)
    keep = O.residual_tokens(s, O.n_residual_tokens(T, ppm))
    Ks = O.candidate_keys(K, O.SHARED, 0)
    contrib = sum(np.sum((Q[l].reshape(-1, d) @ (Ks[l, keep] - K[l, keep]).T) ** 2) / (P * d)
                  for l in range(B)) / (B * G)
    np.testing.assert_allclose(E[O.RESIDUAL], E[O.SHARED] - contrib, rtol=1e-10)
    assert E[O.RESIDUAL] < E[O.SHARED]


@pytest.mark.parametrize("B", [2, 4])
def test_token_unit_reconstruction(B):
    rng = np.random.default_rng(56 + B)
    T, d = 25, 8
    K = rng.standard_normal((B, T, d))
    V = rng.standard_normal((B, T, d))
    tokens = np.array([0, 3, 4, 17, 24])
    unit = O.compress_unit_tokens(K, V, O.RESIDUAL, tokens, "f64")
    assert unit["HK"].shape == (5, B - 1, d)
    mean = K.mean(0)
    for p in range(B):
        Kt = O.reconstruct_layer_tokens(unit, O.RESIDUAL, p, d, "K", B)
        np.testing.assert_allclose(Kt[tokens], K[p, tokens], atol=1e-12)        # kept tokens: exact
        rest = np.setdiff1d(np.arange(T), tokens)
        np.testing.assert_allclose(Kt[rest], mean[rest], atol=1e-12)            # others: the shared mean
        # decode through scipy's inverse DCT of the stored coefficients, brute-force softmax
        Z = np.zeros((B, T, d))
        Z[0] = 2.0 * unit["MK"] if B == 4 else unit["MK"] * math.sqrt(2.0)
        Z[1:, tokens] = np.moveaxis(unit["HK"], 1, 0) if B == 4 else np.moveaxis(unit["HK"], 1, 0) * math.sqrt(2.0)
        np.testing.assert_allclose(scipy.fft.idct(Z, type=2, norm="ortho", axis=0)[p], Kt, atol=1e-12)


def test_token_bytes_closed_form():
    # d = 64, bf16, B = 2, T = 1000, r = 5%: n = 50 tokens
    # M planes 2 * 128000; mask ceil(1000/32)*4 = 128 -> 256; counts (8+1)*4 = 36 -> 256;
    # rows 2 * pad(50 * 64 * 2 = 6400) = 2 * 6400
    assert O.unit_bytes_tokens(O.RESIDUAL, 1000, 64, 50000, "bf16", 2) == 2 * 128000 + 256 + 256 + 2 * 6400
    # fours: three rows per token
    assert O.unit_bytes_tokens(O.RESIDUAL, 1000, 64, 50000, "bf16", 4) == 2 * 128000 + 256 + 256 + 2 * 19200
    assert O.unit_bytes_tokens(O.SHARED, 1000, 64, 50000, "bf16", 4) == O.unit_bytes(O.SHARED, 1000, 64, 0, "bf16", 4)
    np.testing.assert_allclose(O.omega_tokens(128, 50000, "bf16", 2),
                               [0.5, (512 + 2 * 256 * 0.05 + 5 / 32) / 1024, 1.0])


# ---------------------------------------------------------------- token-level sets with per-unit fractions
def test_token_rate_losses_and_costs():
    """E_R(r) at every candidate fraction: E_R(0) = E_S, E_R(1) = 0, non-increasing in r, and
    each equal to the single-fraction loss; Omega of the candidates in closed form."""
    rng = np.random.default_rng(71)
    K = O.round_bf16(rng.standard_normal((2, 60, 16)))
    K[1] = O.round_bf16(0.8 * K[0] + 0.6 * rng.standard_normal((60, 16)))
    Q = O.round_bf16(rng.standard_normal((2, 2, 5, 16)) / 4)
    rates = [0, 20000, 100000, 250000, 1000000]
    E = O.routing_errors_token_rates(K, Q, rates)
    assert E[1] == E[0] and abs(E[-1]) <= 1e-12 * E[0]
    assert np.all(np.diff(E[1:]) <= 1e-15 * E[0])
    for j, r in enumerate(rates):
        assert E[1 + j] == O.routing_errors_tokens(K, Q, r)[O.RESIDUAL]
    om, modes, idx = O.token_rate_candidates(128, [50000, 100000], "bf16", 2)
    np.testing.assert_allclose(om, [512 / 1024, (512 + 25.6 + 1 / 8 + 4 / 128) / 1024,
                                    (512 + 51.2 + 1 / 8 + 4 / 128) / 1024, 1.0], rtol=1e-15)
    assert modes == [O.SHARED, O.RESIDUAL, O.RESIDUAL, O.EXACT] and idx == [0, 0, 1, 0]


def test_token_rate_routing_brute_force():
    """Each unit's (mode, fraction) is the argmin of Eq. (3) over shared, exact and the
    residual mode at every candidate fraction (brute force over the candidates), and the
    budget rule's lambda is the smallest that fits (dense lambda grid), footprint monotone."""
    rng = np.random.default_rng(72)
    T, d, rates = 4000, 64, [10000, 50000, 200000]
    n = 10
    ES = np.abs(rng.standard_normal(n)) * 10
    ER = ES[:, None] * np.sort(rng.uniform(0.05, 0.95, (n, 3)), axis=1)[:, ::-1]    # more tokens, less error
    E = np.concatenate([ES[:, None], ER], axis=1)
    om, cmodes, cidx = O.token_rate_candidates(d, rates, "bf16", 2)
    Ec = np.concatenate([E, np.zeros((n, 1))], axis=1)
    for lam in (0.0, 0.5, 2.0, 5.0, 20.0, 200.0):
        modes, ridx, _, _ = O.route_token_rates(E, T, d, rates, "bf16", lam=lam)
        cost = Ec + lam * om
        best = [min(range(5), key=lambda c: (cost[u, c], om[c])) for u in range(n)]
        np.testing.assert_array_equal(modes, [cmodes[c] for c in best])
        np.testing.assert_array_equal(ridx, [cidx[c] for c in best])

    def fp(lam):
        m, r, _, _ = O.route_token_rates(E, T, d, rates, "bf16", lam=lam)
        return sum(O.unit_bytes_tokens(int(mm), T, d, rates[int(rr)] if mm == O.RESIDUAL else 0, "bf16")
                   for mm, rr in zip(m, r))
    lo, hi = fp(math.inf), fp(0.0)
    for frac in (0.2, 0.5, 0.8):
        budget = int(lo + frac * (hi - lo))
        modes, ridx, lam, ok = O.route_token_rates(E, T, d, rates, "bf16", budget=budget)
        assert ok and fp(lam) <= budget
        assert all(fp(x) > budget for x in np.linspace(0, lam, 1500, endpoint=False))
        lams = np.linspace(0, 3 * lam + 1, 300)
        fps = [fp(x) for x in lams]
        assert all(a >= b for a, b in zip(fps, fps[1:]))
