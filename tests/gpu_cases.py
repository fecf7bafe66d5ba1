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


def unpack_unit(buf: np.ndarray, off: int, mode: int, T: int, d: int, k: int, dtype: str, B: int = 2) -> dict:
    ti, tc = TYPES[dtype]
    e, c = BYTES[ti], BYTES[tc]
    ib = 1 if B == 2 else 2                       # channel bytes (pairs) or uint16 codes 4c + j (fours)
    dense, coef = _pad(T * d * e), _pad(T * d * c)
    ip, vp = _pad(T * k * ib), _pad(T * k * c)

    def plane(o, width, kind):
        return values(buf[off + o: off + o + T * width * BYTES[kind]].copy(), kind).reshape(T, width)

    def index(o):
        raw = buf[off + o: off + o + T * k * ib].copy()
        return (raw if ib == 1 else raw.view("<u2")).astype(np.int64).reshape(T, k)

    if mode == O.EXACT:
        u = {}
        for n in range(B):
            u[f"K{n}"] = plane(n * dense, d, ti)
            u[f"V{n}"] = plane((B + n) * dense, d, ti)
        return u
    u = {"MK": plane(0, d, tc), "MV": plane(coef, d, tc)}
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


def compare_units(gpu_unit: dict, ref_unit: dict, dtype: str, max_ulp: int = 1, inputs=None) -> dict:
    """Per-plane comparison: index and exact planes bit-exact, value planes within ``max_ulp``.

    ``inputs`` = ``(K, V)`` of the unit (``[B][T][d]``) switches fp32 blocks of
    four to an absolute bound: their block mean and butterfly coefficients
    are sums of up to four fp32 products, each rounded, so they sit within
    2^-21 of the largest input magnitude of their channel (plus one unit in
    the last place) of the correctly rounded value the oracle stores.
    """
    stats = {}
    for name, ref in ref_unit.items():
        got = gpu_unit[name]
        assert got.shape == ref.shape, (name, got.shape, ref.shape)
        if name in ("IK", "IV") or (name[0] in "KV" and name[1:].isdigit()):   # indices, exact planes
            np.testing.assert_array_equal(got, ref, err_msg=name)
            stats[name] = 0
            continue
        dist = ulp_distance(got, ref, TYPES[dtype][1])
        if inputs is not None and TYPES[dtype][1] == "f32":
            X = np.asarray(inputs[0 if name[-1] == "K" else 1], np.float64)
            mag = np.abs(X).max(axis=0)                       # [T][d]
            if name[0] == "M":
                bound = mag
            else:
                codes = ref_unit["I" + name[-1]]
                bound = np.take_along_axis(mag, codes >> 2, axis=-1)
            tol = 2.0 ** -21 * bound + np.abs(np.asarray(ref)) * 2.0 ** -23
            bad = np.abs(np.asarray(got) - np.asarray(ref)) > tol
            assert not bad.any(), (name, int(bad.sum()))
        else:
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
