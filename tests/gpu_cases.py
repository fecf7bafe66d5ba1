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


def values(raw: np.ndarray, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return (raw.view(np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return raw.view(np.float32).astype(np.float64)


def unpack_unit(buf: np.ndarray, off: int, mode: int, T: int, d: int, k: int, dtype: str) -> dict:
    e = 4 if dtype == "f32" else 2
    dense = _pad(T * d * e)
    ip, vp = _pad(T * k), _pad(T * k * e)

    def dense_plane(o):
        return values(buf[off + o: off + o + T * d * e].copy(), dtype).reshape(T, d)

    if mode == O.EXACT:
        return {"K0": dense_plane(0), "K1": dense_plane(dense), "V0": dense_plane(2 * dense),
                "V1": dense_plane(3 * dense)}
    u = {"MK": dense_plane(0), "MV": dense_plane(dense)}
    if mode == O.RESIDUAL:
        o = 2 * dense
        u["IK"] = buf[off + o: off + o + T * k].astype(np.int64).reshape(T, k)
        u["VK"] = values(buf[off + o + ip: off + o + ip + T * k * e].copy(), dtype).reshape(T, k)
        o2 = o + ip + vp
        u["IV"] = buf[off + o2: off + o2 + T * k].astype(np.int64).reshape(T, k)
        u["VV"] = values(buf[off + o2 + ip: off + o2 + ip + T * k * e].copy(), dtype).reshape(T, k)
    return u


def ulp_distance(a: np.ndarray, b: np.ndarray, dtype: str) -> np.ndarray:
    """|bit distance| between same-precision values (as ordered integers)."""
    def ordered(x):
        if dtype == "bf16":
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


def compare_units(gpu_unit: dict, ref_unit: dict, dtype: str, max_ulp: int = 1) -> dict:
    """Per-plane comparison: index planes bit-exact, value planes within ``max_ulp``."""
    stats = {}
    for name, ref in ref_unit.items():
        got = gpu_unit[name]
        assert got.shape == ref.shape, (name, got.shape, ref.shape)
        if name in ("IK", "IV"):
            np.testing.assert_array_equal(got, ref, err_msg=name)
            stats[name] = 0
        elif name in ("K0", "K1", "V0", "V1"):
            np.testing.assert_array_equal(got, ref, err_msg=name)
            stats[name] = 0
        else:
            dist = ulp_distance(got, ref, dtype)
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


def oracle_decode_layer(units: dict, modes: np.ndarray, layer: int, q: np.ndarray, w) -> np.ndarray:
    """Oracle output ``[Hq][d]`` of one sequence at ``layer`` (units keyed by (pair, head))."""
    d, G = w.head_dim, w.group
    out = np.zeros((w.n_q_heads, d))
    b = layer // 2
    for h in range(w.n_kv_heads):
        out[h * G:(h + 1) * G] = O.decode_unit(units[(b, h)], int(modes[b, h]), layer,
                                               q[h * G:(h + 1) * G], 1.0 / math.sqrt(d), d)
    return out
