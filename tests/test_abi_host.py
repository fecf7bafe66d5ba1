"""The C-ABI library on the CPU: it loads, exports every declared symbol,
its host-only entry points agree with the oracle, and every validation error
returns before any HIP call (no device work is queued here)."""
import ctypes
import math
import os
import re

import numpy as np
import pytest

import oracle as O
from paper_2607_06519_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B._LIB_PATH):
        pytest.skip("libfdkv.so not built")
    return B.load()


def test_exports_every_declared_symbol(lib):
    hdr = open(os.path.join(ROOT, "include", "fdkv.h")).read()
    declared = set(re.findall(r"\b(fdkv_[a-z_]+)\s*\(", hdr))
    assert declared == set(B.SYMBOLS)
    for name in declared:
        assert hasattr(lib, name)


def test_status_strings(lib):
    for s in (0, -1, -2, -3, -4, -5):
        assert lib.fdkv_status_string(s)
    assert lib.fdkv_last_error() == b""


@pytest.mark.parametrize("dtype,d,k", [("bf16", 128, 16), ("f32", 64, 8), ("bf16", 64, 5), ("f32", 128, 0),
                                     ("bf16_e4m3", 128, 16), ("bf16_e4m3", 64, 5)])
def test_layout_matches_oracle(lib, dtype, d, k):
    rng = np.random.default_rng(d + k)
    L, H, batch = 6, 3, 4
    dm = B.dims(L, H, 2 * H, d, k, dtype)
    seq = rng.integers(0, 3000, size=batch)
    seq[1] = 1
    modes = rng.integers(0, 3, size=(batch, L // 2, H)).astype(np.uint8)
    off, total = B.layout(dm, seq, modes)
    assert total == O.cache_bytes(seq, modes, d, k, dtype)
    # offsets are the running sums of the oracle's per-unit bytes
    sizes = [O.unit_bytes(int(m), int(seq[b]), d, k, dtype) for b in range(batch) for m in modes[b].ravel()]
    np.testing.assert_array_equal(off.ravel(), np.concatenate([[0], np.cumsum(sizes)[:-1]]))
    assert (off % 256 == 0).all()


def test_layout_tiny_closed_form(lib):
    dm = B.dims(2, 4, 4, 64, 8, "f32")
    _, total = B.layout(dm, [512], np.array([[[0, 1, 1, 2]]], np.uint8))
    assert total == 1392640


def _rand_errors(rng, units):
    E = np.abs(rng.standard_normal((units, 2))).astype(np.float32) * 50
    E[:, 1] = (E[:, 0] * rng.uniform(0.3, 0.7, units)).astype(np.float32)
    return E


@pytest.mark.parametrize("dtype,d,k", [("bf16", 128, 16), ("f32", 64, 8), ("bf16_e4m3", 128, 16)])
def test_route_lambda_matches_oracle(lib, dtype, d, k):
    rng = np.random.default_rng(5)
    dm = B.dims(32, 8, 32, d, k, dtype)
    E = _rand_errors(rng, 128)
    E3 = np.concatenate([E.astype(np.float64), np.zeros((128, 1))], axis=1)
    om = O.omega(d, k, dtype)
    for lam in (0.0, 1.0, 7.5, 33.0, 1e9):
        modes, lam_used, st = B.route(dm, 32768, E.reshape(16, 8, 2), lam=lam)
        assert st == 0 and lam_used == lam
        np.testing.assert_array_equal(modes.ravel(), O.route(E3, om, lam))


def test_route_at_breakpoints_matches_oracle(lib):
    """At every unit's own breakpoints the C rule and the oracle give the same
    modes (the tie goes to the cheaper mode on both sides)."""
    rng = np.random.default_rng(9)
    d, k = 128, 16
    dm = B.dims(32, 8, 32, d, k, "bf16")
    E = _rand_errors(rng, 128)
    E3 = np.concatenate([E.astype(np.float64), np.zeros((128, 1))], axis=1)
    om = O.omega(d, k, "bf16")
    for u in range(0, 128, 9):
        for a, b in ((0, 1), (1, 2), (0, 2)):
            lam = (E3[u, a] - E3[u, b]) / (om[b] - om[a])
            modes, _, st = B.route(dm, 32768, E.reshape(16, 8, 2), lam=float(lam))
            assert st == 0
            np.testing.assert_array_equal(modes.ravel(), O.route(E3, om, lam))


@pytest.mark.parametrize("frac", [0.0, 0.15, 0.5, 0.85, 1.0])
def test_route_budget_matches_oracle(lib, frac):
    rng = np.random.default_rng(6)
    d, k, T = 128, 16, 32768
    dm = B.dims(32, 8, 32, d, k, "bf16")
    E = _rand_errors(rng, 128)
    E3 = np.concatenate([E.astype(np.float64), np.zeros((128, 1))], axis=1)
    lo = 128 * O.unit_bytes(O.SHARED, T, d, k, "bf16")
    hi = 128 * O.unit_bytes(O.EXACT, T, d, k, "bf16")
    budget = int(lo + frac * (hi - lo))
    modes, lam, st = B.route(dm, T, E.reshape(16, 8, 2), budget_bytes=budget)
    om_modes, om_lam, ok = O.route_budget(E3, T, d, k, "bf16", budget)
    assert st == 0 and ok
    np.testing.assert_array_equal(modes.ravel(), om_modes)
    assert lam == om_lam


def test_route_budget_infeasible(lib):
    dm = B.dims(4, 2, 2, 64, 8, "bf16")
    E = np.ones((2, 2, 2), np.float32)
    modes, lam, st = B.route(dm, 100, E, budget_bytes=1, allow_infeasible=True)
    assert st == -4 and (modes == 0).all() and math.isinf(lam)


def test_validation_errors_before_any_device_call(lib):
    """Invalid arguments return the right status; the fake pointers are never used."""
    good = B.dims(4, 2, 8, 128, 16, "bf16")
    fake = ctypes.c_void_p(1 << 20)          # aligned, never dereferenced
    ptrs = (ctypes.c_void_p * 4)(*([1 << 20] * 4))
    st = lambda d, **kw: lib.fdkv_decode_attn(ctypes.byref(d), kw.get("batch", 1), fake, 16, fake, fake, fake,
                                              kw.get("layer", 0), fake, fake, ctypes.c_float(0.1), fake,
                                              kw.get("ws", 0), None)
    assert st(good) == -3                                   # workspace too small
    assert st(good, layer=4) == -1
    assert st(good, batch=0) == -1
    assert st(B.dims(3, 2, 8, 128, 16, "bf16")) == -1      # odd layers
    assert st(B.dims(4, 2, 7, 128, 16, "bf16")) == -1      # Hq not a multiple of Hkv
    assert st(B.dims(4, 2, 8, 96, 16, "bf16")) == -2       # head_dim not compiled
    assert st(B.dims(4, 1, 16, 128, 16, "bf16")) == -2     # group of 16
    assert st(B.dims(4, 2, 8, 128, 129, "bf16")) == -1     # k > d
    assert st(B.dims(4, 2, 8, 128, 16, 7)) == -1           # dtype
    mis = ctypes.c_void_p((1 << 20) + 4)
    assert lib.fdkv_decode_attn(ctypes.byref(good), 1, fake, 16, fake, fake, fake, 0, mis, fake,
                                ctypes.c_float(0.1), fake, 1 << 30, None) == -1
    odd = ctypes.c_void_p((1 << 20) + 1)                   # modes are read in aligned 4-byte words
    assert lib.fdkv_decode_attn(ctypes.byref(good), 1, fake, 16, odd, fake, fake, 0, fake, fake,
                                ctypes.c_float(0.1), fake, 1 << 30, None) == -1
    # planes are addressed with 32-bit offsets: T * d * 2 bytes must stay below 2^31
    assert lib.fdkv_decode_attn(ctypes.byref(good), 1, fake, 1 << 23, fake, fake, fake, 0, fake, fake,
                                ctypes.c_float(0.1), fake, 1 << 40, None) == -2
    assert lib.fdkv_compress(ctypes.byref(good), 16, ptrs, None, fake, fake, None, None, fake, None) == -1
    n = ctypes.c_size_t(0)
    assert lib.fdkv_probe_workspace(ctypes.byref(good), 100, 4, ctypes.byref(n)) == 0 and n.value > 0
    assert lib.fdkv_probe(ctypes.byref(good), 100, ptrs, ptrs, 4, fake, None, fake, n.value - 1, None, None) == -3
    assert lib.fdkv_probe(ctypes.byref(good), 0, ptrs, ptrs, 4, fake, None, fake, n.value, None, None) == -1
    assert lib.fdkv_probe(ctypes.byref(good), 1 << 23, ptrs, ptrs, 4, fake, None, fake, 1 << 40, None, None) == -2
    # the K selection buffer: one byte per 16-byte input piece of every unit's rows
    sb = ctypes.c_size_t(0)
    assert lib.fdkv_selection_bytes(ctypes.byref(good), 100, ctypes.byref(sb)) == 0
    assert sb.value == (good.n_layers // 2) * good.n_kv_heads * 100 * (good.head_dim * 2 // 16)
    assert lib.fdkv_selection_bytes(ctypes.byref(good), -1, ctypes.byref(sb)) == -1
    mixed = B.dims(12, 2, 8, 128, 16, "bf16", schedule=B.MIXED)     # blocks 2,2,4,2,2: 4-byte slots
    assert lib.fdkv_selection_bytes(ctypes.byref(mixed), 100, ctypes.byref(sb)) == 0
    assert sb.value == 5 * 2 * 100 * 16 * 4
    assert lib.fdkv_selection_bytes(ctypes.byref(good), 100, None) == -1
    assert lib.fdkv_layout(None, 1, None, None, None, None) == -1


# ---------------------------------------------------------------- block schedules
@pytest.mark.parametrize("L,sched", [(32, B.MIXED), (8, B.MIXED), (12, B.MIXED), (16, B.QUADS), (4, B.QUADS),
                                     (6, B.PAIRS), (128, B.MIXED)])
def test_blocks_match_oracle(lib, L, sched):
    first, size = B.blocks(B.dims(L, 2, 4, 64, 8, "bf16", sched))
    want = O.block_schedule(L, sched)
    assert list(zip(first.tolist(), size.tolist())) == [tuple(x) for x in want]


def test_schedule_validation(lib):
    n = ctypes.c_int32(0)
    for L, sched in [(10, B.MIXED), (6, B.MIXED), (6, B.QUADS), (7, B.PAIRS), (8, 3), (8, -1), (130, B.PAIRS)]:
        assert lib.fdkv_blocks(ctypes.byref(B.dims(L, 2, 4, 64, 8, "bf16", sched)), ctypes.byref(n), None, None) == -1


@pytest.mark.parametrize("dtype,d,k,sched", [("bf16", 128, 16, B.MIXED), ("f32", 64, 8, B.QUADS),
                                             ("bf16_e4m3", 128, 16, B.MIXED), ("bf16", 64, 5, B.QUADS),
                                             ("f32", 128, 0, B.MIXED)])
def test_layout_blocks_match_oracle(lib, dtype, d, k, sched):
    rng = np.random.default_rng(d + k + 7 * sched)
    L, H, batch = 12, 3, 3
    dm = B.dims(L, H, 2 * H, d, k, dtype, sched)
    sizes = [Bs for _, Bs in O.block_schedule(L, sched)]
    seq = rng.integers(0, 3000, size=batch)
    seq[1] = 1
    modes = rng.integers(0, 3, size=(batch, len(sizes), H)).astype(np.uint8)
    off, total = B.layout(dm, seq, modes)
    assert total == O.cache_bytes(seq, modes, d, k, dtype, sizes)
    unit = [O.unit_bytes(int(modes[b, i, h]), int(seq[b]), d, k, dtype, sizes[i])
            for b in range(batch) for i in range(len(sizes)) for h in range(H)]
    np.testing.assert_array_equal(off.ravel(), np.concatenate([[0], np.cumsum(unit)[:-1]]))


@pytest.mark.parametrize("frac", [0.0, 0.2, 0.6, 1.0])
def test_route_budget_mixed_matches_oracle(lib, frac):
    rng = np.random.default_rng(60)
    d, k, T, H = 128, 16, 32768, 8
    dm = B.dims(32, H, 32, d, k, "bf16", B.MIXED)
    sizes = [Bs for _, Bs in O.block_schedule(32, O.MIXED)]
    usz = [Bs for Bs in sizes for _ in range(H)]
    n = len(usz)
    E = _rand_errors(rng, n)
    E3 = np.concatenate([E.astype(np.float64), np.zeros((n, 1))], axis=1)
    lo = sum(O.unit_bytes(O.SHARED, T, d, k, "bf16", Bs) for Bs in usz)
    hi = sum(O.unit_bytes(O.EXACT, T, d, k, "bf16", Bs) for Bs in usz)
    budget = int(lo + frac * (hi - lo))
    modes, lam, st = B.route(dm, T, E.reshape(len(sizes), H, 2), budget_bytes=budget)
    om_modes, om_lam, ok = O.route_budget(E3, T, d, k, "bf16", budget, usz)
    assert st == 0 and ok
    np.testing.assert_array_equal(modes.ravel(), om_modes)
    assert lam == om_lam
    for lam_fixed in (0.0, 3.0, 40.0):
        om = np.stack([O.omega(d, k, "bf16", Bs) for Bs in usz])
        m2, _, _ = B.route(dm, T, E.reshape(len(sizes), H, 2), lam=lam_fixed)
        np.testing.assert_array_equal(m2.ravel(), O.route(E3, om, lam_fixed))


def test_generation_entry_points_validate(lib):
    good = B.dims(4, 2, 8, 128, 16, "bf16")
    fake = ctypes.c_void_p(1 << 20)
    n = ctypes.c_size_t(0)
    m = (ctypes.c_int32 * 3)(1000, 513, 0)
    assert lib.fdkv_decode_spans_workspace(ctypes.byref(good), 2, 3, m, 64, ctypes.byref(n)) == 0
    # chunks of 512 tokens: 2 + 2 + 0 spans + 1 tail, per (sequence, KV head), G = 4, d + 4 floats
    assert n.value == 2 * 2 * 5 * 4 * 132 * 4
    assert lib.fdkv_decode_spans_workspace(ctypes.byref(good), 2, 16, (ctypes.c_int32 * 16)(), 64, ctypes.byref(n)) == -1
    assert lib.fdkv_decode_spans_workspace(ctypes.byref(good), 2, 16, (ctypes.c_int32 * 16)(), -1, ctypes.byref(n)) == 0
    sp = (B.Span * 1)(B.Span(1 << 20, 16, 1 << 20, 1 << 20, 1 << 20))
    tl = B.Tail(1 << 20, 8, 1 << 20, 1 << 20)
    call = lambda spans, tail, **kw: lib.fdkv_decode_spans(ctypes.byref(good), 1, kw.get("n", 1), spans, tail,
                                                          kw.get("layer", 0), fake, fake, ctypes.c_float(0.1), fake,
                                                          kw.get("ws", 0), None)
    assert call(ctypes.cast(sp, ctypes.c_void_p), ctypes.byref(tl)) == -3          # workspace too small
    assert call(ctypes.cast(sp, ctypes.c_void_p), ctypes.byref(tl), layer=4) == -1
    assert call(None, ctypes.byref(tl), n=1) == -1                                  # spans missing
    bad = (B.Span * 1)(B.Span(1 << 20, 16, (1 << 20) + 1, 1 << 20, 1 << 20))      # modes not 4-byte aligned
    assert call(ctypes.cast(bad, ctypes.c_void_p), None, ws=1 << 30) == -1
    big = B.Tail(1 << 20, 1 << 23, 1 << 20, 1 << 20)                                 # cap * d * 2 >= 2^31
    assert call(ctypes.cast(sp, ctypes.c_void_p), ctypes.byref(big), ws=1 << 40) == -2
    assert lib.fdkv_append(ctypes.byref(good), 1, fake, 0, fake, fake, fake, fake, None) == -1     # cap 0
    assert lib.fdkv_append(ctypes.byref(good), 1, ctypes.c_void_p((1 << 20) + 2), 8, fake, fake, fake, fake,
                           None) == -1


# ---------------------------------------------------------------- token-level residual set
@pytest.mark.parametrize("dtype,d,ppm,sched", [("bf16", 128, 50000, B.PAIRS), ("f32", 64, 123456, B.QUADS),
                                               ("bf16_e4m3", 128, 1000000, B.MIXED), ("bf16", 64, 0, B.MIXED)])
def test_layout_tokens_match_oracle(lib, dtype, d, ppm, sched):
    rng = np.random.default_rng(ppm % 97 + d)
    L, H, batch = 12, 2, 3
    dm = B.dims(L, H, 2 * H, d, 0, dtype, sched, B.RES_TOKENS, ppm)
    sizes = [Bs for _, Bs in O.block_schedule(L, sched)]
    seq = rng.integers(0, 5000, size=batch)
    seq[0] = 1
    modes = rng.integers(0, 3, size=(batch, len(sizes), H)).astype(np.uint8)
    off, total = B.layout(dm, seq, modes)
    unit = [O.unit_bytes_tokens(int(modes[b, i, h]), int(seq[b]), d, ppm, dtype, sizes[i])
            for b in range(batch) for i in range(len(sizes)) for h in range(H)]
    assert total == sum(unit)
    np.testing.assert_array_equal(off.ravel(), np.concatenate([[0], np.cumsum(unit)[:-1]]))


def test_route_tokens_matches_oracle(lib):
    rng = np.random.default_rng(61)
    d, T, H, ppm = 128, 32768, 8, 50000
    dm = B.dims(32, H, 32, d, 0, "bf16", B.MIXED, B.RES_TOKENS, ppm)
    usz = [Bs for _, Bs in O.block_schedule(32, O.MIXED) for _ in range(H)]
    E = _rand_errors(rng, len(usz))
    E3 = np.concatenate([E.astype(np.float64), np.zeros((len(usz), 1))], axis=1)
    om = np.stack([O.omega_tokens(d, ppm, "bf16", Bs) for Bs in usz])
    for lam in (0.0, 2.0, 17.0, 1e9):
        m, _, _ = B.route(dm, T, E.reshape(-1, H, 2), lam=lam)
        np.testing.assert_array_equal(m.ravel(), O.route(E3, om, lam))


def test_tokens_validation(lib):
    n = ctypes.c_int32(0)
    for ppm in (-1, 1000001):
        bad = B.dims(4, 2, 4, 64, 0, "bf16", B.PAIRS, B.RES_TOKENS, ppm)
        assert lib.fdkv_blocks(ctypes.byref(bad), ctypes.byref(n), None, None) == -1
    bad = B.dims(4, 2, 4, 64, 0, "bf16", B.PAIRS, 2, 0)
    assert lib.fdkv_blocks(ctypes.byref(bad), ctypes.byref(n), None, None) == -1


def test_static_decode_checks_its_scratch_on_the_host(lib):
    """fdkv_decode_attn_static refuses a call whose split-K records exceed its static
    scratch, and bad dimensions, before any HIP call (the fake pointers are never used)."""
    fake = ctypes.c_void_p(1 << 20)
    big = B.dims(2, 8, 64, 128, 16, "bf16")
    need = ctypes.c_size_t(0)
    assert lib.fdkv_decode_workspace(ctypes.byref(big), 4, 131072, ctypes.byref(need)) == 0
    assert need.value > lib.fdkv_decode_static_scratch_bytes() == 16 << 20
    st = lib.fdkv_decode_attn_static(ctypes.byref(big), 4, fake, 131072, fake, fake, fake, 0, fake, fake,
                                     ctypes.c_float(0.1), None)
    assert st == -3 and b"static scratch" in lib.fdkv_last_error()
    bad = B.dims(2, 8, 64, 96, 16, "bf16")
    assert lib.fdkv_decode_attn_static(ctypes.byref(bad), 1, fake, 100, fake, fake, fake, 0, fake, fake,
                                       ctypes.c_float(0.1), None) == -2


def test_route_with_routed_fractions_matches_oracle(lib):
    """Token-level sets with per-unit fractions: fdkv_route over (mode, fraction) candidates
    equals the oracle's route_token_rates at several lambdas and under budgets, and
    fdkv_layout prices each unit at its own fraction."""
    rng = np.random.default_rng(13)
    rates = (10000, 50000, 200000)
    J, T, d = len(rates), 4096, 128
    dm = B.dims(8, 2, 8, d, 0, "bf16", residual=B.RES_TOKENS, res_rates=rates)
    n = 4 * 2
    ES = np.abs(rng.standard_normal(n)).astype(np.float32) * 20
    ER = (ES[:, None] * np.sort(rng.uniform(0.05, 0.95, (n, J)), axis=1)[:, ::-1]).astype(np.float32)
    E = np.concatenate([ES[:, None], ER], axis=1)                          # [units][1 + J]
    for lam in (0.0, 1.0, 5.0, 30.0, 1e9):
        modes, _, st = B.route(dm, T, E.reshape(4, 2, 1 + J), lam=lam)
        assert st == 0
        om_m, om_r, _, _ = O.route_token_rates(E.astype(np.float64), T, d, rates, "bf16", lam=lam)
        np.testing.assert_array_equal(modes.ravel() & 3, om_m)
        np.testing.assert_array_equal((modes.ravel() >> 2)[om_m == 1], om_r[om_m == 1])
        assert np.all((modes.ravel() >> 2)[om_m != 1] == 0)
    lo = n * O.unit_bytes_tokens(O.SHARED, T, d, 0, "bf16")
    hi = n * O.unit_bytes_tokens(O.EXACT, T, d, 0, "bf16")
    for frac in (0.1, 0.3, 0.6):
        budget = int(lo + frac * (hi - lo))
        modes, lam, st = B.route(dm, T, E.reshape(4, 2, 1 + J), budget_bytes=budget)
        om_m, om_r, om_lam, ok = O.route_token_rates(E.astype(np.float64), T, d, rates, "bf16", budget=budget)
        assert st == 0 and ok and lam == om_lam
        np.testing.assert_array_equal(modes.ravel() & 3, om_m)
        np.testing.assert_array_equal((modes.ravel() >> 2)[om_m == 1], om_r[om_m == 1])
        offs, total = B.layout(dm, [T], modes[None])
        want = sum(O.unit_bytes_tokens(int(m), T, d, rates[int(r)] if m == 1 else 0, "bf16")
                   for m, r in zip(om_m, om_r))
        assert total == want <= budget


def test_mode_bytes_are_validated(lib):
    """A fraction index only on a residual unit of a cache with that many routed fractions."""
    good = B.dims(2, 1, 1, 64, 0, "bf16", residual=B.RES_TOKENS, res_rates=(10000, 20000))
    plain = B.dims(2, 1, 1, 64, 4, "bf16")
    assert B.layout(good, [100], np.array([[[1 | (1 << 2)]]], np.uint8))[1] > 0
    for dm, byte in ((good, 1 | (2 << 2)), (good, 2 | (1 << 2)), (good, 0 | (1 << 2)), (good, 3),
                     (plain, 1 | (1 << 2)), (good, 1 | (1 << 5))):
        total = ctypes.c_uint64(0)
        modes = np.array([byte], np.uint8)
        lens = np.array([100], np.int32)
        st = lib.fdkv_layout(ctypes.byref(dm), 1, lens.ctypes.data_as(ctypes.c_void_p),
                             modes.ctypes.data_as(ctypes.c_void_p), None, ctypes.byref(total))
        assert st == -1, byte
    # routed fractions need token-level sets, increasing and within 0..10^6
    for dm in (B.dims(2, 1, 1, 64, 4, "bf16", res_rates=(1000,)),
               B.dims(2, 1, 1, 64, 0, "bf16", residual=B.RES_TOKENS, res_rates=(2000, 1000)),
               B.dims(2, 1, 1, 64, 0, "bf16", residual=B.RES_TOKENS, res_rates=(2000, 2000000))):
        n = ctypes.c_int32(0)
        assert lib.fdkv_blocks(ctypes.byref(dm), ctypes.byref(n), None, None) == -1
