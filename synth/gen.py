"""Seeded draws for the synthetic workloads.

Every array comes from its own ``numpy`` PCG64 substream keyed by
``SeedSequence([seed, cfg_id, tag, ...])``, so any (sequence, layer pair, KV
head) segment can be regenerated on its own, in any order and on any host.

Recipe of one (sequence, block, KV head h) segment of B layers, for K and for
V alike (a first-order autoregression along depth):

* ``x[l0] ~ N(0, 1)`` per token and channel;
* ``x[l+1] = rho * x[l] + sqrt(1 - rho^2) * eps`` with ``eps ~ N(0, 1)``,
  one ``rho ~ U(lo, hi)`` per segment shared by K and V, independent ``eps``;
* needle tokens (positions drawn once per sequence) get ``+amp`` on a seeded
  set of distinct channels in one layer of the block (the last layer, or a
  seeded choice per needle), the same channels and layer for K and V;
* values are finally rounded to the storage precision (bf16 round to
  nearest even, or kept as fp32).

All returned arrays are ``float32`` holding values exactly representable in
the workload's storage type.
"""
from __future__ import annotations

import math
from concurrent.futures import ThreadPoolExecutor
from typing import Iterator, Tuple

import numpy as np

from .workloads import Workload

_TAG_SEGMENT, _TAG_POS, _TAG_DECODE_Q, _TAG_PROBE_Q, _TAG_MODES, _TAG_SEGMENT4 = 1, 2, 3, 4, 5, 6


def _rng(w: Workload, *tags: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([w.seed, w.cfg_id, *tags])))


def round_bf16_f32(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 (ties to even), returned as float32 values."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    bias = ((u >> np.uint32(16)) & np.uint32(1)) + np.uint32(0x7FFF)
    r = (u + bias) & np.uint32(0xFFFF0000)
    return r.view(np.float32)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are exactly bfloat16 (as uint16)."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    return (u >> np.uint32(16)).astype(np.uint16)


def to_storage(x: np.ndarray, dtype: str) -> np.ndarray:
    x = np.asarray(x, dtype=np.float32)
    if dtype in ("bf16", "bf16_e4m3"):  # the FP8-coefficient cache type takes bf16 inputs
        return round_bf16_f32(x)
    if dtype == "f32":
        return np.ascontiguousarray(x)
    raise ValueError(f"unknown dtype {dtype!r}")


def needle_positions(w: Workload, seq: int) -> np.ndarray:
    T = w.seq_lens[seq]
    n = min(w.n_needles, T)
    rng = _rng(w, _TAG_POS, seq)
    return np.sort(rng.choice(T, size=n, replace=False)).astype(np.int64)


def segment(w: Workload, seq: int, pair: int, head: int):
    """K and V of one (sequence, pair, KV head) segment.

    Returns ``(K, V, info)`` with ``K, V`` of shape ``[2][T][d]`` (layer 2b
    then 2b+1) and ``info`` holding ``rho`` and the needle plan
    ``[(position, layer, channels), ...]``.
    """
    T, d = w.seq_lens[seq], w.head_dim
    rng = _rng(w, _TAG_SEGMENT, seq, pair, head)
    lo, hi = w.rho
    rho = float(lo) if lo == hi else float(rng.uniform(lo, hi))
    c1 = np.float32(rho)
    c2 = np.float32(math.sqrt(1.0 - rho * rho))
    out = []
    for _ in range(2):  # K, then V
        x0 = rng.standard_normal((T, d), dtype=np.float32)
        eps = rng.standard_normal((T, d), dtype=np.float32)
        x = np.empty((2, T, d), dtype=np.float32)
        x[0] = x0
        np.multiply(x0, c1, out=x[1])
        x[1] += c2 * eps
        out.append(x)
    K, V = out
    plan = []
    for pos in needle_positions(w, seq):
        if w.needle_layer == "odd":
            layer = 1
        elif w.needle_layer == "coin":
            layer = int(rng.integers(0, 2))
        else:
            raise ValueError(w.needle_layer)
        ch = np.sort(rng.choice(d, size=min(w.needle_channels, d), replace=False))
        K[layer, pos, ch] += np.float32(w.needle_amp)
        V[layer, pos, ch] += np.float32(w.needle_amp)
        plan.append((int(pos), layer, ch))
    K = to_storage(K, w.dtype)
    V = to_storage(V, w.dtype)
    return K, V, {"rho": rho, "needles": plan}


def block_segment(w: Workload, seq: int, block: int, head: int):
    """K and V ``[B][T][d]`` of one (sequence, block, KV head) segment of the workload's schedule.

    A pair is the segment of ``segment`` (keyed by its pair index); a block of
    four draws a four-layer chain from its own substream.
    """
    first, B = w.blocks[block]
    if B == 2:
        return segment(w, seq, first // 2, head)
    T, d = w.seq_lens[seq], w.head_dim
    rng = _rng(w, _TAG_SEGMENT4, seq, first, head)
    lo, hi = w.rho
    rho = float(lo) if lo == hi else float(rng.uniform(lo, hi))
    c1 = np.float32(rho)
    c2 = np.float32(math.sqrt(1.0 - rho * rho))
    out = []
    for _ in range(2):  # K, then V
        x = np.empty((B, T, d), dtype=np.float32)
        x[0] = rng.standard_normal((T, d), dtype=np.float32)
        for n in range(1, B):
            np.multiply(x[n - 1], c1, out=x[n])
            x[n] += c2 * rng.standard_normal((T, d), dtype=np.float32)
        out.append(x)
    K, V = out
    plan = []
    for pos in needle_positions(w, seq):
        layer = B - 1 if w.needle_layer == "odd" else int(rng.integers(0, B))
        ch = np.sort(rng.choice(d, size=min(w.needle_channels, d), replace=False))
        K[layer, pos, ch] += np.float32(w.needle_amp)
        V[layer, pos, ch] += np.float32(w.needle_amp)
        plan.append((int(pos), layer, ch))
    return to_storage(K, w.dtype), to_storage(V, w.dtype), {"rho": rho, "needles": plan}


def iter_segments(w: Workload, seq: int, threads: int = 8) -> Iterator[Tuple[int, int, np.ndarray, np.ndarray]]:
    """Yield ``(block, head, K, V)`` for every segment of one sequence, drawn in parallel."""
    units = [(b, h) for b in range(w.n_blocks) for h in range(w.n_kv_heads)]

    def one(u):
        K, V, _ = block_segment(w, seq, u[0], u[1])
        return u[0], u[1], K, V

    if threads <= 1:
        for u in units:
            yield one(u)
        return
    with ThreadPoolExecutor(max_workers=threads) as ex:
        # bounded look-ahead keeps host memory to a few segments
        pending = []
        it = iter(units)
        for u in it:
            pending.append(ex.submit(one, u))
            if len(pending) >= 2 * threads:
                yield pending.pop(0).result()
        for f in pending:
            yield f.result()


def layer_cache(w: Workload, seq: int = 0, threads: int = 1):
    """Whole cache of one sequence as ``K, V`` of shape ``[L][Hkv][T][d]``."""
    L, H, T, d = w.n_layers, w.n_kv_heads, w.seq_lens[seq], w.head_dim
    K = np.empty((L, H, T, d), dtype=np.float32)
    V = np.empty((L, H, T, d), dtype=np.float32)
    for b, h, k, v in iter_segments(w, seq, threads):
        first, B = w.blocks[b]
        K[first:first + B, h] = k
        V[first:first + B, h] = v
    return K, V


def decode_queries(w: Workload, step: int, scale: float = 1.0) -> np.ndarray:
    """Decode queries of one step, ``[L][batch][Hq][d]`` ~ N(0,1)/sqrt(d) times ``scale``."""
    rng = _rng(w, _TAG_DECODE_Q, step)
    q = rng.standard_normal((w.n_layers, w.batch, w.n_q_heads, w.head_dim), dtype=np.float32)
    q *= np.float32(scale / math.sqrt(w.head_dim))
    return to_storage(q, w.dtype)


def probe_queries(w: Workload, seq: int = 0, layers=None) -> np.ndarray:
    """Probe-window queries ``[L][Hq][P][d]`` ~ N(0,1)/sqrt(d) (one substream per layer)."""
    layers = range(w.n_layers) if layers is None else layers
    P, d = w.n_probe, w.head_dim
    out = np.empty((len(layers), w.n_q_heads, P, d), dtype=np.float32)
    for i, l in enumerate(layers):
        rng = _rng(w, _TAG_PROBE_Q, seq, l)
        out[i] = rng.standard_normal((w.n_q_heads, P, d), dtype=np.float32)
    out *= np.float32(1.0 / math.sqrt(d))
    return to_storage(out, w.dtype)


def fixed_modes(w: Workload, seq: int = 0) -> np.ndarray:
    """Head modes ``[blocks][Hkv]`` (0 shared, 1 residual, 2 exact) for decode timing.

    Either the workload's explicit list, or a seeded shuffle of its
    shared/residual/exact counts (scaled to the number of units).
    """
    n = w.n_blocks * w.n_kv_heads
    if w.fixed_modes is not None:
        m = np.asarray(w.fixed_modes, dtype=np.uint8)
        if m.size != n:
            m = np.resize(m, n)
        return m.reshape(w.n_blocks, w.n_kv_heads)
    if w.mode_counts is None:
        raise ValueError(f"workload {w.name} has no fixed modes")
    cs, cr, ce = w.mode_counts
    scale = n / float(cs + cr + ce)
    ns, nr = int(round(cs * scale)), int(round(cr * scale))
    ne = n - ns - nr
    m = np.array([0] * ns + [1] * nr + [2] * ne, dtype=np.uint8)
    rng = _rng(w, _TAG_MODES, seq)
    rng.shuffle(m)
    return m.reshape(w.n_blocks, w.n_kv_heads)
