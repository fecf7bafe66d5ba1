"""Shared helpers of the GPU parity tests: seeded inputs to device tensors,
the GPU path through the C ABI, and reading the packed cache back into the
oracle's per-unit format (the layout documented in include/fdkv.h, re-read
here independently of the library)."""
from __future__ import annotations

import math

import numpy as np

import oracle as O
from synth import gen

PLANE = 256


def _pad(n):
    return -(-n // PLANE) * PLANE


# OCP FP8 E4M3 decoding of the 256 codes (sign, 4 exponent bits with bias 7,
# 3 mantissa bits, subnormals, S.1111.111 = NaN), from the format definition
_codes = np.arange(256)
_e, _m = (_codes >> 3) & 15, _codes & 7
_mag = np.where(_e == 0, _m * 2.0 ** -9, (1.0 + _m / 8.0) * 2.0 ** (_e - 7.0))
_mag = np.where((_e == 15) & (_m == 7), np.nan, _mag)
E4M3 = np.where(_codes >= 128, -_mag, _mag)
_E4M3_POS = np.sort(_mag[:127])          # finite non-negative values, ascending (0 .. 448)

# cache type -> (input / exact-plane type, coefficient type)
TYPES = {"f32": ("f32", "f32"), "bf16": ("bf16", "bf16"), "bf16_e4m3": ("bf16", "e4m3")}
BYTES = {"f32": 4, "bf16": 2, "e4m3": 1}


def values(raw: np.ndarray, kind: str) -> np.ndarray:
    if kind == "bf16":
        return (raw.view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    if kind == "e4m3":
        return E4M3[raw]
    return raw.view(np.float32).astype(np.float64)


def coef_plane_bytes(T: int, d: int, c: int) -> int:
    """A shared plane's bytes: FP8 planes fill whole 1 KB blocks."""
    return _pad(-(-(T * d) // 1024) * 1024) if c == 1 else _pad(T * d * c)


def shared_plane(buf: np.ndarray, o: int, T: int, d: int, dtype: str) -> np.ndarray:
    """A shared (M) plane ``[T][d]`` read back from byte ``o``.  FP8 planes (the
    layout of include/fdkv.h): 1 KB blocks of R = 1024 / d rows; rows t and
    t + R/2 of a block share each 16-byte slot, slot (t % (R/2)) * d/8 + p
    holding channels 8p .. 8p + 7 of the first row, then of the second."""
    tc = TYPES[dtype][1]
    if BYTES[tc] != 1:
        return values(buf[o: o + T * d * BYTES[tc]].copy(), tc).reshape(T, d)
    R, npc = 1024 // d, d // 8
    t = np.arange(T)[:, None]
    p = np.arange(npc)[None, :]
    at = (t // R) * 1024 + 16 * ((t % (R // 2)) * npc + p) + 8 * ((t % R) // (R // 2))
    raw = buf[o + at[..., None] + np.arange(8)]
    return values(raw.reshape(-1).copy(), tc).reshape(T, d)


def unpack_unit(buf: np.ndarray, off: int, mode: int, T: int, d: int, k: int, dtype: str, B: int = 2) -> dict:
    ti, tc = TYPES[dtype]
    e, c = BYTES[ti], BYTES[tc]
    ib = 1 if B == 2 else 2                       # channel bytes (pairs) or uint16 codes 4c + j (fours)
    fp8 = c == 1
    dense = _pad(T * d * e)
    coef = coef_plane_bytes(T, d, c)
    ip, vp = _pad(T * k * ib), _pad(T * k * c)

    def plane(o, width, kind):
        return values(buf[off + o: off + o + T * width * BYTES[kind]].copy(), kind).reshape(T, width)

    def block_plane(o):
        return shared_plane(buf, off + o, T, d, dtype)

    def index(o):
        raw = buf[off + o: off + o + T * k * ib].copy()
        return (raw if ib == 1 else raw.view("<u2")).astype(np.int64).reshape(T, k)

    if mode == O.EXACT:
        u = {}
        for n in range(B):
            u[f"K{n}"] = plane(n * dense, d, ti)
            u[f"V{n}"] = plane((B + n) * dense, d, ti)
        return u
    u = {"MK": block_plane(0), "MV": block_plane(coef)} if fp8 else {"MK": plane(0, d, tc), "MV": plane(coef, d, tc)}
    if mode == O.RESIDUAL:
        o = 2 * coef
        u["IK"] = index(o)
        u["VK"] = plane(o + ip, k, tc)
        o2 = o + ip + vp
        u["IV"] = index(o2)
        u["VV"] = plane(o2 + ip, k, tc)
    return u


def ulp_distance(a: np.ndarray, b: np.ndarray, kind: str) -> np.ndarray:
    """|bit distance| between same-precision values (as ordered integers)."""
    def ordered(x):
        x = np.asarray(x, np.float64)
        if kind == "e4m3":
            i = np.searchsorted(_E4M3_POS, np.abs(x)).astype(np.int64)
            return np.where(x < 0, -i, i)
        if kind == "bf16":
            u = (np.asarray(x, np.float32).view(np.uint32) >> 16).astype(np.int64)
            sign = 0x8000
        else:
            u = np.asarray(x, np.float32).view(np.uint32).astype(np.int64)
            sign = 0x80000000
        return np.where(u & sign, -(u & (sign - 1)), u)
    return np.abs(ordered(a) - ordered(b))


def rel_l2(a, b) -> float:
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    n = np.linalg.norm(b)
    return float(np.linalg.norm(a - b) / (n if n > 0 else 1.0))


# significant bits of each coefficient type, and its smallest spacing (subnormals)
_SIG_BITS = {"f32": 24, "bf16": 8, "e4m3": 4}
_MIN_SPACING = {"f32": 2.0 ** -149, "bf16": 2.0 ** -133, "e4m3": 2.0 ** -9}
QUAD_BAND = 2.0 ** -21     # fp32 DCT-II(4) butterfly error, relative to the channel's largest input


def quad_value_tol(ref: np.ndarray, mag: np.ndarray, kind: str) -> np.ndarray:
    """Allowed |stored - oracle| for a coefficient of a block of four: the fp32
    butterfly or block mean sits within 2^-21 of the channel's largest input
    magnitude ``mag`` of the exact value (the bound derived in
    test_dct4_host.py), and the rounding to the storage type adds at most one
    spacing of that type at the value."""
    ref = np.abs(np.asarray(ref, np.float64))
    return QUAD_BAND * mag + ref * 2.0 ** (1 - _SIG_BITS[kind]) + _MIN_SPACING[kind]


def check_quad_codes(got_codes: np.ndarray, X: np.ndarray, k: int, what: str = "") -> int:
    """Residual codes of a block of four (``[T][k]`` uint16 ``4 c + j``, ascending) against
    the oracle's float64 ranking of |Z_j[c]| (Eq. 1).  The kernel ranks the fp32
    butterfly's values, which sit within 2^-21 M (M: the token's largest input
    magnitude) of the exact ones, so: every code whose key clears the k-th largest key
    by more than twice that band is taken, none below it by as much is, and each token
    takes k distinct valid codes in ascending order.  Returns the number of tokens whose
    set differs from the oracle's (all such differences lie inside the band)."""
    X = np.asarray(X, np.float64)
    T, d = X.shape[1], X.shape[2]
    got = np.asarray(got_codes, np.int64).reshape(T, k)
    if k == 0:
        return 0
    key = O.residual_keys_dct4(X).reshape(T, 3 * d)              # position 3 c + j - 1
    j, c = got & 3, got >> 2
    assert np.all((j >= 1) & (c < d)), what
    assert np.all(np.diff(got, axis=1) > 0), what                   # ascending, distinct
    taken = np.zeros((T, 3 * d), bool)
    np.put_along_axis(taken, 3 * c + j - 1, True, axis=1)
    band = 2.0 * QUAD_BAND * np.abs(X).max(axis=(0, 2))[:, None]   # [T][1]
    tau = np.sort(key, axis=1)[:, -k][:, None]
    assert not np.any((key > tau + band) & ~taken), what
    assert not np.any((key < tau - band) & taken), what
    want = O.residual_codes_dct4(X, k)
    wtaken = np.zeros((T, 3 * d), bool)
    np.put_along_axis(wtaken, 3 * (want >> 2) + (want & 3) - 1, True, axis=1)
    return int(np.any(taken != wtaken, axis=1).sum())


def compare_units(gpu_unit: dict, ref_unit: dict, dtype: str, max_ulp: int = 1, inputs=None) -> dict:
    """Per-plane comparison.  Pairs: index and exact planes bit-exact, value
    planes within ``max_ulp``.  Blocks of four (``inputs`` = ``(K, V)`` of the
    unit, ``[4][T][d]``): exact planes bit-exact, residual codes by the
    near-tie rule of ``check_quad_codes``, values at the kernel's codes and the
    block mean within ``quad_value_tol`` of the oracle's (float64 rounded to the
    storage type)."""
    stats = {}
    quad = inputs is not None and np.asarray(inputs[0]).shape[0] == 4
    kind = TYPES[dtype][1]
    for name, ref in ref_unit.items():
        got = gpu_unit[name]
        assert got.shape == ref.shape, (name, got.shape, ref.shape)
        if name[0] in "KV" and name[1:].isdigit():                  # exact planes
            np.testing.assert_array_equal(got, ref, err_msg=name)
            stats[name] = 0
            continue
        if name in ("IK", "IV"):
            if quad:
                X = np.asarray(inputs[0 if name == "IK" else 1], np.float64)
                stats[name + "_band"] = check_quad_codes(got, X, got.shape[-1], name)
            else:
                np.testing.assert_array_equal(got, ref, err_msg=name)
                stats[name] = 0
            continue
        if quad:
            X = np.asarray(inputs[0 if name[-1] == "K" else 1], np.float64)
            mag = np.abs(X).max(axis=0)                                # [T][d]
            if name[0] == "M":
                want = ref
            else:                                                     # values at the kernel's codes
                codes = np.asarray(gpu_unit["I" + name[-1]], np.int64)
                Z = O.depth_factorize(X)
                t = np.arange(X.shape[1])[:, None]
                want = O.round_coef(Z[codes & 3, t, codes >> 2], dtype)
                mag = np.take_along_axis(mag, codes >> 2, axis=-1)
            bad = np.abs(np.asarray(got, np.float64) - want) > quad_value_tol(want, mag, kind)
            assert not bad.any(), (name, int(bad.sum()))
            stats[name] = int((ulp_distance(got, want, kind) > 0).sum())
            continue
        dist = ulp_distance(got, ref, kind)
        assert dist.max(initial=0) <= max_ulp, (name, int(dist.max()))
        stats[name] = int((dist > 0).sum())
    return stats


def sharpened_queries(w, step: int, K: np.ndarray, scales=(1.0, 8.0, 32.0)):
    """Decode queries at several sharpness levels plus one aligned with a needle key.

    Returns a list of ``[L][batch][Hq][d]`` float32 arrays of storage values.
    """
    out = [gen.decode_queries(w, step, scale=s) for s in scales]
    # needle-aligned: each query head points at the key of its KV head at the
    # first needle position, scaled to make that token dominate
    pos = gen.needle_positions(w, 0)
    if len(pos):
        q = np.zeros_like(out[0])
        G = w.group
        for l in range(w.n_layers):
            for hq in range(w.n_q_heads):
                key = K[l, hq // G, pos[0]].astype(np.float64)
                q[l, 0, hq] = key / (np.linalg.norm(key) + 1e-12) * 4.0
        out.append(gen.to_storage(q, w.dtype))
    return out


def block_of(w, layer: int):
    """``(block index, first layer, B)`` of ``layer`` in the workload's schedule."""
    for i, (first, B) in enumerate(w.blocks):
        if first <= layer < first + B:
            return i, first, B
    raise ValueError(layer)


def oracle_decode_layer(units: dict, modes: np.ndarray, layer: int, q: np.ndarray, w) -> np.ndarray:
    """Oracle output ``[Hq][d]`` of one sequence at ``layer`` (units keyed by (block, head))."""
    d, G = w.head_dim, w.group
    out = np.zeros((w.n_q_heads, d))
    b, _, B = block_of(w, layer)
    for h in range(w.n_kv_heads):
        out[h * G:(h + 1) * G] = O.decode_unit(units[(b, h)], int(modes[b, h]), layer,
                                               q[h * G:(h + 1) * G], 1.0 / math.sqrt(d), d, B)
    return out


# ---------------------------------------------------------------- head modes against the oracle's routing
NEAR_TIE = 1e-4     # relative cost margin below which a unit's mode is a near-tie


def cost_margins(E3: np.ndarray, om: np.ndarray, lam: float):
    """The oracle's modes at ``lam`` and each unit's relative cost margin: the
    smallest (cost of another mode - cost of the chosen one) / cost of the chosen
    one (inf when the chosen cost is 0)."""
    om = np.asarray(om, np.float64)
    C = om.shape[-1]
    E3 = np.asarray(E3, np.float64).reshape(-1, C)
    om = np.broadcast_to(om, E3.shape)
    modes = O.route(E3, om, lam)
    cost = E3 + lam * om if np.isfinite(lam) else np.where(om == om.min(axis=1, keepdims=True), 0.0, np.inf)
    marg = np.empty(len(E3))
    for u, m in enumerate(modes):
        c = cost[u, m]
        other = min(cost[u, j] for j in range(C) if j != m)
        marg[u] = other / c - 1.0 if c > 0 else np.inf
    return modes, marg


def breakpoints(E3: np.ndarray, om: np.ndarray) -> np.ndarray:
    """Every positive breakpoint (E_a - E_b) / (O_b - O_a), a the cheaper candidate, sorted."""
    om = np.asarray(om, np.float64)
    E3 = np.asarray(E3, np.float64).reshape(-1, om.shape[-1])
    return np.array(O.breakpoint_candidates(E3, np.broadcast_to(om, E3.shape)))


def separated_lambdas(E3: np.ndarray, om: np.ndarray, n: int = 3) -> list:
    """``n`` penalties at the midpoints between consecutive breakpoints, spread over
    the breakpoint list: there every mode decision is as far from a tie as the
    data allows."""
    bp = breakpoints(E3, om)
    if len(bp) < 2:
        return [float(bp[0]) * 0.5] if len(bp) else [1.0]
    idx = np.unique(np.linspace(0, len(bp) - 2, n).round().astype(int))
    return [float(0.5 * (bp[i] + bp[i + 1])) for i in idx]


def check_modes(got_modes, E3, om, lam: float, what: str = "", exclude=(), near: float = NEAR_TIE) -> int:
    """Head modes bit-exact against the oracle's at ``lam``; units whose oracle
    cost margin is below NEAR_TIE are near-ties, reported and required to be
    absent (``exclude`` lists units tied by construction, e.g. the unit whose
    breakpoint a budget lambda is).  Returns the number of units compared."""
    want, marg = cost_margins(E3, om, lam)
    got = np.asarray(got_modes).ravel()
    mask = np.ones(len(want), bool)
    mask[list(exclude)] = False
    tie = near
    near = np.nonzero(mask & (marg < tie))[0]
    print(f"    modes {what} at lambda {lam:.6g}: {int(mask.sum())} units, near-ties {near.tolist()}, "
          f"smallest margin {marg[mask].min(initial=np.inf):.3g}", flush=True)
    assert near.size == 0, (what, lam, near, marg[near])
    np.testing.assert_array_equal(got[mask], want[mask], err_msg=f"{what} lambda {lam}")
    return int(mask.sum())


def budget_defining_units(E3, om, lam: float) -> list:
    """Units with a breakpoint equal to ``lam`` (two of their candidates tie there)."""
    om = np.asarray(om, np.float64)
    C = om.shape[-1]
    E3 = np.asarray(E3, np.float64).reshape(-1, C)
    om = np.broadcast_to(om, E3.shape)
    out = []
    for u in range(len(E3)):
        for i in range(C):
            for j in range(i + 1, C):
                a, b = (i, j) if om[u, i] <= om[u, j] else (j, i)
                if om[u, b] > om[u, a] and (E3[u, a] - E3[u, b]) / (om[u, b] - om[u, a]) == lam:
                    out.append(u)
    return sorted(set(out))
