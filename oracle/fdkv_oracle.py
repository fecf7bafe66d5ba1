"""Plain CPU oracle of the FreqDepthKV compressed-cache path (fp64 numpy).

TEST INFRASTRUCTURE ONLY.  Only the tests, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this module.  It shares no code
with the GPU path (no kernels, headers, helpers or table generators); both
sides only share the seeded input generator in ``synth``.

Everything is computed in float64 straight from the method's definitions in
the paper (Section 3, "Method"), slowly and without any blocking or fusion:

* depth factorization, Eq. (1): ``Z = F_B X`` and ``X = F_B^T Z`` with an
  orthonormal DCT-II basis ``F_B`` along the layer axis of a block;
* compressed representation, Eq. (3): the low-frequency coefficient is kept
  for every token, the high-frequency coefficients only on a residual set
  (empty for shared-depth heads, everything for exact heads);
* routing loss, Eq. (2): the mean over probe queries of the squared norm of
  the difference between the logit rows under the reconstructed and the
  original keys, plus ``lambda * Omega(m)``; ``m = argmin`` over the three
  modes (Eq. 3), the budget rule raising ``lambda`` until the footprint fits
  (end of Section 3);
* decode attention over the reconstructed K/V (Section 3, the paragraph after
  Eq. 3), a full softmax with max subtraction;
* token-level residual set (Section 3, after Eq. 2): residual heads keep every
  high-frequency coefficient of the ``r T`` tokens with the largest score
  ``s_t = max_q |q (K_t - K^S_t)^T|``;
* generation (the end of Section 3's method): tokens produced while decoding
  are kept exact in a tail; a refresh compresses the tail into a new span of
  the cache, routed by Eq. (2) on the tail's own keys with the most recent
  decode queries as probe rows; decode attends over every span and the tail.

Readings of the paper adopted here (the paper leaves these open):

* blocks are adjacent layer pairs (B = 2) and ``F_2`` is the orthonormal
  DCT-II, i.e. the Haar matrix ``[[1, 1], [1, -1]] / sqrt(2)``; the mixed
  schedule of Section 4 puts B = 4 blocks (``F_4``, the orthonormal
  DCT-II(4)) between B = 2 blocks covering the first and the last four
  layers (``block_schedule``);
* the residual keeps, for every token, the ``k`` channels of largest
  ``|x[2b] - x[2b+1]|`` (computed in float32 on the stored inputs; ties go to
  the lower channel; indices stored ascending), K and V chosen independently;
* what is stored is the per-layer image of each coefficient, ``P_k X`` with
  the projector ``P_k = F[k]^T F[k]``: ``M`` (the pair mean) for k = 0 and
  ``D`` (half the difference) for k = 1, so layer 2b reconstructs ``M + D``
  and layer 2b+1 ``M - D``; the projector entries are evaluated in 50-digit
  decimal arithmetic so that stored values are correctly rounded;
* in a B = 4 block the residual of a token keeps the ``k`` largest of its
  ``3 d`` high-frequency coefficients ``|Z_j[c]|`` (j = 1..3; by Parseval this
  minimises the block's squared reconstruction error), ranked by their
  float64 values (``residual_keys_dct4``), ties to the lower code
  ``4 c + j``; what is stored
  is the code (uint16, ascending) and the orthonormal coefficient ``Z_j[c]``
  itself, and layer ``p`` of the block adds ``F_4[j, p] Z_j[c]``; the shared
  plane is the image of ``Z_0``, the four-layer mean;
* the routing loss of a (block, KV head) averages Eq. (2) over the layers of
  the block and over the query heads of the KV head's group, uses the
  unrounded coefficients (storage rounding is not part of the method), and
  leaves values to follow the keys' decision;
* ``Omega(m)`` is the bytes per token of mode ``m`` divided by those of exact
  mode; ties in the argmin go to the cheaper mode;
* the budget rule takes the smallest ``lambda`` among 0, the per-head
  breakpoints and +inf whose footprint fits the budget;
* decode scales logits by ``1/sqrt(d)`` and attends over the cached tokens;
* the token score is computed in float64 from the stored inputs; its
  maximum runs over the probe rows of every layer of the block and every
  query head of the group; ``r`` is one fraction per cache (parts per
  million), ``n = ceil(r T)``, ties to the lower token; the stored rows are
  the unrounded coefficients rounded to the coefficient type;
* with several candidate fractions, each residual (block, head) takes its own
  fraction: every fraction is one more candidate of Eq. (3)'s argmin (its
  loss E_R(r) and its Omega), and the budget rule runs over all candidates
  (``route_token_rates``);
* a refresh re-decides routing only for the tokens it compresses (earlier
  spans keep their modes: a shared head's dropped coefficients cannot be
  recovered), and a span's probe rows are the last decode queries;
* cache type ``bf16_e4m3`` (the quantised-coefficient variant the paper
  allows at the end of Section 3): inputs, queries and exact heads are bf16;
  the shared and residual coefficients (``M`` and the residual values) are
  stored in OCP FP8 E4M3, rounded once, to nearest with ties to even, from
  the unrounded coefficient, saturating at +-448; no scale factor.

Parity status: every function here is pinned by tests against closed forms,
textbook routines, brute force and a hand-worked example, except that no
value printed in the paper can be reproduced (it gives no worked example).
"""
from __future__ import annotations

import functools
import math
from typing import Dict, Tuple

import numpy as np

SHARED, RESIDUAL, EXACT = 0, 1, 2
MODES = (SHARED, RESIDUAL, EXACT)
PLANE_ALIGN = 256

_BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127
_E4M3_MAX = 448.0
# cache types: bytes and rounding of the input (exact-head) planes and of the coefficient planes
_INPUT_TYPE = {"f32": "f32", "bf16": "bf16", "bf16_e4m3": "bf16"}
_COEF_TYPE = {"f32": "f32", "bf16": "bf16", "bf16_e4m3": "e4m3"}
_TYPE_BYTES = {"f32": 4, "bf16": 2, "e4m3": 1, "f64": 8}


def input_bytes(dtype: str) -> int:
    """Bytes per element of the inputs and of exact-head planes."""
    return _TYPE_BYTES[_INPUT_TYPE.get(dtype, dtype)]


def coef_bytes(dtype: str) -> int:
    """Bytes per element of the stored shared / residual coefficients."""
    return _TYPE_BYTES[_COEF_TYPE.get(dtype, dtype)]


# ----------------------------------------------------------------------------
# storage precision
# ----------------------------------------------------------------------------
def round_bf16(x) -> np.ndarray:
    """Nearest bfloat16 value (round half to even), computed from float64."""
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)                       # |x| = m * 2**e with m in [0.5, 1)
    q = np.maximum(e - 8, -133)              # 8 significant bits; subnormal quantum 2**-133
    y = np.ldexp(np.round(np.ldexp(x, -q)), q)
    return np.where(np.abs(y) > _BF16_MAX, np.copysign(np.inf, x), y)


def round_e4m3(x) -> np.ndarray:
    """Nearest OCP FP8 E4M3 value (round half to even), saturating at +-448.

    E4M3 has 4 significant bits for normal values (|x| >= 2**-6) and a
    subnormal quantum of 2**-9; 480 and above have no finite encoding, so the
    largest finite value 448 absorbs everything beyond it.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)                       # |x| = m * 2**e with m in [0.5, 1)
    q = np.maximum(e - 4, -9)                # 4 significant bits; subnormal quantum 2**-9
    y = np.ldexp(np.round(np.ldexp(x, -q)), q)
    return np.where(np.abs(y) > _E4M3_MAX, np.copysign(_E4M3_MAX, x), y)


def round_to_storage(x, dtype: str) -> np.ndarray:
    x = np.asarray(x, dtype=np.float64)
    if dtype == "f64":
        return x.copy()
    if dtype == "f32":
        return x.astype(np.float32).astype(np.float64)
    if dtype == "bf16":
        return round_bf16(x)
    if dtype == "e4m3":
        return round_e4m3(x)
    raise ValueError(dtype)


def round_input(x, dtype: str) -> np.ndarray:
    """Rounding of the inputs / exact-head planes of a cache type."""
    return round_to_storage(x, _INPUT_TYPE.get(dtype, dtype))


def round_coef(x, dtype: str) -> np.ndarray:
    """Rounding of the stored shared / residual coefficients of a cache type."""
    return round_to_storage(x, _COEF_TYPE.get(dtype, dtype))


# ----------------------------------------------------------------------------
# Eq. (1): depth factorization
# ----------------------------------------------------------------------------
def dct_matrix(B: int) -> np.ndarray:
    """Orthonormal DCT-II basis F_B (rows = frequencies, columns = layers).

    ``F[k, n] = s_k cos(pi (2n+1) k / (2B))`` with ``s_0 = sqrt(1/B)`` and
    ``s_k = sqrt(2/B)``, each entry evaluated in 50-digit decimal arithmetic
    and rounded once to float64 (so ``F_4[2] = [1/2, -1/2, -1/2, 1/2]``
    exactly and the mirror symmetry ``F[k, B-1-n] = (-1)^k F[k, n]`` holds
    bit for bit).
    """
    return _dct_matrix_cached(B).copy()


@functools.lru_cache(maxsize=None)
def _dct_matrix_cached(B: int) -> np.ndarray:
    import decimal
    prec = 50
    with decimal.localcontext() as ctx:
        ctx.prec = prec + 10
        pi = _dec_pi(prec)
        F = np.empty((B, B), dtype=np.float64)
        for k in range(B):
            s = (decimal.Decimal(1 if k == 0 else 2) / B).sqrt()
            for n in range(B):
                F[k, n] = float(s * _dec_cos(pi * (2 * n + 1) * k / (2 * B), prec))
    return F


def _dec_pi(prec: int):
    """pi to ``prec`` decimal digits (Machin's formula)."""
    import decimal
    with decimal.localcontext() as ctx:
        ctx.prec = prec + 10

        def arctan_inv(x):
            x = decimal.Decimal(x)
            total, term, n, sign = decimal.Decimal(0), 1 / x, 1, 1
            x2 = x * x
            while term > decimal.Decimal(10) ** -(prec + 5):
                total += sign * term / n
                term /= x2
                n += 2
                sign = -sign
            return total

        return +(16 * arctan_inv(5) - 4 * arctan_inv(239))


def _dec_cos(x, prec: int):
    """cos of a Decimal by its Taylor series (|x| small after reduction)."""
    import decimal
    with decimal.localcontext() as ctx:
        ctx.prec = prec + 10
        pi = _dec_pi(prec)
        x = x % (2 * pi)
        total, term, n = decimal.Decimal(1), decimal.Decimal(1), 0
        while abs(term) > decimal.Decimal(10) ** -(prec + 5):
            n += 2
            term = -term * x * x / (n * (n - 1))
            total += term
        return +total


@functools.lru_cache(maxsize=None)
def _dct_projectors_cached(B: int) -> np.ndarray:
    return _dct_projectors_exact(B)


def dct_projectors(B: int) -> np.ndarray:
    """Per-layer images of each DCT coefficient (see ``_dct_projectors_exact``)."""
    return _dct_projectors_cached(B).copy()


def _dct_projectors_exact(B: int) -> np.ndarray:
    """Per-layer images of each DCT coefficient: ``P[k, l, n] = F[k, l] F[k, n]``.

    ``P_k X`` is the part of the block ``X`` carried by frequency ``k`` (Eq. 1:
    ``X = F^T Z = sum_k F[k]^T F[k] X``).  The products are evaluated in
    50-digit decimal arithmetic and rounded once to float64, so for B = 2 they
    are exactly +-1/2 and the stored images come out correctly rounded.
    """
    import decimal
    prec = 50
    with decimal.localcontext() as ctx:
        ctx.prec = prec + 10
        pi = _dec_pi(prec)
        P = np.empty((B, B, B), dtype=np.float64)
        for k in range(B):
            s2 = decimal.Decimal(1 if k == 0 else 2) / B
            for l in range(B):
                cl = _dec_cos(pi * (2 * l + 1) * k / (2 * B), prec)
                for n in range(B):
                    cn = _dec_cos(pi * (2 * n + 1) * k / (2 * B), prec)
                    P[k, l, n] = float(s2 * cl * cn)
    return P


def coefficient_image(X, k: int, layer: int) -> np.ndarray:
    """Layer ``layer``'s share of DCT coefficient ``k`` of the block ``X``: ``sum_n P[k,l,n] x_n``."""
    X = np.asarray(X, dtype=np.float64)
    P = dct_projectors(X.shape[0])
    out = np.zeros_like(X[0])
    for n in range(X.shape[0]):
        out += P[k, layer, n] * X[n]
    return out


def depth_factorize(X) -> np.ndarray:
    """Z = F_B X along the leading (layer) axis of a block.

    Terms are grouped by the mirror symmetry ``F[k, B-1-n] = (-1)^k F[k, n]``:
    ``Z_k = sum_{n < B/2} F[k, n] (x_n + (-1)^k x_{B-1-n})`` (plus the middle
    layer when B is odd), the same sum in exact arithmetic; with it, identical
    or mirror-symmetric layers give exactly zero coefficients.
    """
    X = np.asarray(X, dtype=np.float64)
    B = X.shape[0]
    F = dct_matrix(B)
    Z = np.zeros_like(X)
    for k in range(B):
        sign = 1.0 if k % 2 == 0 else -1.0
        for n in range(B // 2):
            Z[k] += F[k, n] * (X[n] + sign * X[B - 1 - n])
        if B % 2:
            Z[k] += F[k, B // 2] * X[B // 2]
    return Z


def depth_reconstruct(Z) -> np.ndarray:
    """X = F_B^T Z along the leading (frequency) axis."""
    Z = np.asarray(Z, dtype=np.float64)
    F = dct_matrix(Z.shape[0])
    X = np.zeros_like(Z)
    for n in range(Z.shape[0]):
        for k in range(Z.shape[0]):
            X[n] += F[k, n] * Z[k]
    return X


# ----------------------------------------------------------------------------
# block schedules (Section 4: B = 4 by default, B = 2 for the first and the
# last four layers)
# ----------------------------------------------------------------------------
PAIRS, MIXED, QUADS = 0, 1, 2
SCHEDULES = (PAIRS, MIXED, QUADS)


def block_schedule(n_layers: int, schedule: int = PAIRS):
    """``[(first layer, B), ...]`` of the blocks covering layers ``0 .. L-1`` in order.

    PAIRS: every block a pair.  QUADS: every block four layers.  MIXED (the
    paper's default setting): two pairs, then blocks of four, then two pairs.
    """
    L = int(n_layers)
    if schedule == PAIRS:
        ok, sizes = L >= 2 and L % 2 == 0, [2] * (L // 2)
    elif schedule == QUADS:
        ok, sizes = L >= 4 and L % 4 == 0, [4] * (L // 4)
    elif schedule == MIXED:
        ok, sizes = L >= 8 and (L - 8) % 4 == 0, [2, 2] + [4] * ((L - 8) // 4) + [2, 2]
    else:
        raise ValueError(f"schedule {schedule}")
    if not ok:
        raise ValueError(f"{L} layers do not fit schedule {schedule}")
    out, first = [], 0
    for B in sizes:
        out.append((first, B))
        first += B
    return out


def block_of_layer(n_layers: int, schedule: int, layer: int) -> Tuple[int, int, int]:
    """``(block index, B, position of the layer in its block)``."""
    for i, (first, B) in enumerate(block_schedule(n_layers, schedule)):
        if first <= layer < first + B:
            return i, B, layer - first
    raise ValueError(f"layer {layer}")


# ----------------------------------------------------------------------------
# residual channel set (per token top-k of |x[2b] - x[2b+1]|)
# ----------------------------------------------------------------------------
def residual_keys(x_even, x_odd) -> np.ndarray:
    """|fl32(x[2b] - x[2b+1])|: the ranking key, in float32 arithmetic."""
    a = np.asarray(x_even, dtype=np.float32)
    b = np.asarray(x_odd, dtype=np.float32)
    return np.abs(a - b)


def residual_channels(x_even, x_odd, k: int) -> np.ndarray:
    """Ascending channel indices ``[..., k]`` of the k largest keys per token.

    Ties go to the lower channel index.
    """
    key = residual_keys(x_even, x_odd)
    d = key.shape[-1]
    if k == 0:
        return np.zeros(key.shape[:-1] + (0,), dtype=np.int64)
    chan = np.broadcast_to(np.arange(d), key.shape)
    order = np.lexsort((chan, -key), axis=-1)      # key descending, then channel ascending
    return np.sort(order[..., :k], axis=-1).astype(np.int64)


def residual_keys_dct4(X) -> np.ndarray:
    """Ranking keys ``|Z_j[c]|``, j = 1..3, of a B = 4 block, ``[..., d, 3]``.

    ``X``: ``[4][..., d]`` stored inputs of the block's layers.  The keys are the
    magnitudes of the high-frequency coefficients ``Z = F_4 X`` of Eq. (1), in
    float64 (``depth_factorize``).
    """
    Z = depth_factorize(np.asarray(X, dtype=np.float64))
    return np.abs(np.moveaxis(Z[1:], 0, -1))


def residual_codes_dct4(X, k: int) -> np.ndarray:
    """Ascending codes ``4 c + j`` ``[..., k]`` of the k largest keys per token (ties to the lower code)."""
    key = residual_keys_dct4(X)
    d = key.shape[-2]
    key = key.reshape(key.shape[:-2] + (3 * d,))        # position 3 c + (j - 1): code order
    pos = np.arange(3 * d)
    code = 4 * (pos // 3) + pos % 3 + 1
    if k == 0:
        return np.zeros(key.shape[:-1] + (0,), dtype=np.int64)
    order = np.lexsort((np.broadcast_to(pos, key.shape), -key), axis=-1)
    return code[np.sort(order[..., :k], axis=-1)].astype(np.int64)


# ----------------------------------------------------------------------------
# Eq. (3): compressed representation of one (block, KV head) unit
# ----------------------------------------------------------------------------
def compress_unit(KB, VB, mode: int, k: int, dtype: str) -> Dict[str, np.ndarray]:
    """Stored planes of one unit.

    ``KB, VB``: ``[B][T][d]`` inputs of the block's layers (B = 2 or 4).
    Returns a dict with ``MK, MV`` ([T][d], the image of the low-frequency
    coefficient) for shared/residual heads, plus ``IK, VK, IV, VV`` ([T][k]
    indices and values) for residual heads, or ``K0 .. K{B-1}, V0 ..`` (the
    inputs) for exact heads.  B = 2: indices are channels and values the
    half difference ``D`` at them.  B = 4: indices are codes ``4 c + j`` and
    values the coefficients ``Z_j[c]``.  Values are rounded to the storage
    precision.
    """
    B = len(KB)
    if B not in (2, 4):
        raise ValueError(f"block size {B}")
    out: Dict[str, np.ndarray] = {}
    if mode == EXACT:
        for name, X in (("K", KB), ("V", VB)):
            X = np.asarray(X, dtype=np.float64)
            for n in range(B):
                out[name + str(n)] = round_input(X[n], dtype)
        return out
    for name, X in (("K", KB), ("V", VB)):
        X = np.asarray(X, dtype=np.float64)
        out["M" + name] = round_coef(coefficient_image(X, 0, 0), dtype)
        if mode != RESIDUAL:
            continue
        if B == 2:
            idx = residual_channels(X[0], X[1], k)
            D = coefficient_image(X, 1, 0)
            out["I" + name] = idx
            out["V" + name] = round_coef(np.take_along_axis(D, idx, axis=-1), dtype)
        else:
            codes = residual_codes_dct4(X, k)
            Z = depth_factorize(X)
            t = np.arange(X.shape[1])[:, None]
            out["I" + name] = codes
            out["V" + name] = round_coef(Z[codes & 3, t, codes >> 2], dtype)
    return out


def reconstruct_layer(unit: Dict[str, np.ndarray], mode: int, pos: int, d: int, which: str,
                      B: int = 2) -> np.ndarray:
    """K~ or V~ (``which`` = "K"/"V") of layer ``pos`` of a B-layer block from the stored planes (Eq. 3)."""
    if mode == EXACT:
        return np.asarray(unit[which + str(pos)], dtype=np.float64)
    F = dct_matrix(B)
    M = np.asarray(unit["M" + which], dtype=np.float64)
    T = M.shape[0]
    Z = np.zeros((B, T, d), dtype=np.float64)
    Z[0] = M / F[0, 0]
    if mode == RESIDUAL and unit["I" + which].shape[-1] > 0:
        idx = np.asarray(unit["I" + which])
        vals = np.asarray(unit["V" + which], dtype=np.float64)
        if B == 2:
            np.put_along_axis(Z[1], idx, vals / F[1, 0], axis=-1)
        else:
            t = np.broadcast_to(np.arange(T)[:, None], idx.shape)
            Z[idx & 3, t, idx >> 2] = vals
    return depth_reconstruct(Z)[pos]


# ----------------------------------------------------------------------------
# decode attention over the reconstructed cache
# ----------------------------------------------------------------------------
def attention(q, K, V, scale: float) -> np.ndarray:
    """softmax(q K^T * scale) V for q ``[G][d]``, K, V ``[T][d]`` (fp64, max-subtracted)."""
    q = np.asarray(q, dtype=np.float64)
    s = (q @ np.asarray(K, dtype=np.float64).T) * scale
    s = s - s.max(axis=-1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=-1, keepdims=True)
    return p @ np.asarray(V, dtype=np.float64)


def decode_unit(unit, mode: int, layer: int, q, scale: float, d: int, B: int = 2) -> np.ndarray:
    """Output rows ``[G][d]`` of the G query heads of one KV head at ``layer``.

    ``layer mod B`` is the layer's position in its block: every schedule
    starts a block of B layers at a multiple of B.
    """
    pos = layer % B
    Kt = reconstruct_layer(unit, mode, pos, d, "K", B)
    Vt = reconstruct_layer(unit, mode, pos, d, "V", B)
    return attention(q, Kt, Vt, scale)


# ----------------------------------------------------------------------------
# token-level residual set (Section 3, the paragraph after Eq. 2): a residual
# head keeps every high-frequency coefficient of its top r*T tokens, ranked by
# the largest logit change the token's removal would cause at a probe row
# ----------------------------------------------------------------------------
def token_deviations(KB) -> np.ndarray:
    """Deviations ``K_t - K^S_t`` of each layer's keys from the shared
    reconstruction, ``[B][T][d]``, in float64 on the stored inputs: ``x_l - M``
    with ``M`` the block mean (pairs: ``(x0 - x1) / 2`` and its negation)."""
    X = np.asarray(KB, dtype=np.float64)
    return X - coefficient_image(X, 0, 0)[None]


def token_scores(KB, QB) -> Tuple[np.ndarray, np.ndarray]:
    """``(s, e)`` per token: ``s_t = max |q . dev_{l,t}|`` over the probe rows q of every
    layer l of the block and every query head of the group, and ``e_t`` the sum of
    the squares of those dot products (float64)."""
    dev = token_deviations(KB)
    QB = np.asarray(QB, dtype=np.float64)
    s = np.zeros(dev.shape[1])
    e = np.zeros(dev.shape[1])
    for l in range(dev.shape[0]):
        Q = QB[l].reshape(-1, QB.shape[-1])                 # [G*P][d]
        L = Q @ dev[l].T                                     # [G*P][T]
        s = np.maximum(s, np.abs(L).max(axis=0))
        e += (L * L).sum(axis=0)
    return s, e


def n_residual_tokens(T: int, ppm: int) -> int:
    """r*T rounded up, r = ppm / 10^6."""
    return (int(T) * int(ppm) + 999999) // 1000000


def residual_tokens(scores, n: int) -> np.ndarray:
    """Ascending indices of the ``n`` highest scores, ties to the lower token."""
    scores = np.asarray(scores, dtype=np.float64)
    if n == 0:
        return np.zeros(0, dtype=np.int64)
    order = np.lexsort((np.arange(scores.size), -scores))
    return np.sort(order[:n]).astype(np.int64)


def compress_unit_tokens(KB, VB, mode: int, tokens, dtype: str) -> Dict[str, np.ndarray]:
    """Stored planes of one unit with a token-level residual set ``tokens``.

    Shared / exact heads are as in ``compress_unit``.  A residual head stores
    ``MK, MV`` plus, for its tokens (ascending, ``TS``), every high-frequency
    coefficient of K and V: ``HK, HV`` of shape ``[n][B-1][d]`` (pairs: the half
    difference D; fours: Z_1..Z_3), rounded to the coefficient type.
    """
    if mode != RESIDUAL:
        return compress_unit(KB, VB, mode, 0, dtype)
    out = compress_unit(KB, VB, SHARED, 0, dtype)
    tokens = np.asarray(tokens, dtype=np.int64)
    out["TS"] = tokens
    B = len(KB)
    for name, X in (("K", KB), ("V", VB)):
        X = np.asarray(X, dtype=np.float64)
        if B == 2:
            H = coefficient_image(X, 1, 0)[tokens][:, None, :]
        else:
            H = np.moveaxis(depth_factorize(X)[1:, tokens], 0, 1)
        out["H" + name] = round_coef(H, dtype)
    return out


def reconstruct_layer_tokens(unit, mode: int, pos: int, d: int, which: str, B: int = 2) -> np.ndarray:
    """K~ or V~ of layer ``pos`` of a block from a token-level residual unit (Eq. 3)."""
    if mode != RESIDUAL:
        return reconstruct_layer(unit, mode, pos, d, which, B)
    F = dct_matrix(B)
    M = np.asarray(unit["M" + which], dtype=np.float64)
    Z = np.zeros((B,) + M.shape)
    Z[0] = M / F[0, 0]
    tokens = unit["TS"]
    H = np.asarray(unit["H" + which], dtype=np.float64)
    if B == 2:
        Z[1, tokens] = H[:, 0] / F[1, 0]
    else:
        Z[1:, tokens] = np.moveaxis(H, 1, 0)
    return depth_reconstruct(Z)[pos]


def decode_unit_tokens(unit, mode: int, layer: int, q, scale: float, d: int, B: int = 2) -> np.ndarray:
    pos = layer % B
    return attention(q, reconstruct_layer_tokens(unit, mode, pos, d, "K", B),
                     reconstruct_layer_tokens(unit, mode, pos, d, "V", B), scale)


def routing_errors_tokens(KB, QB, ppm: int) -> np.ndarray:
    """Eq. (2) for the three modes with the token-level residual: the residual
    reconstruction keeps every high-frequency coefficient of the ``ppm``-fraction
    of tokens with the highest scores (unrounded coefficients)."""
    KB = np.asarray(KB, dtype=np.float64)
    QB = np.asarray(QB, dtype=np.float64)
    T, d = KB.shape[1], KB.shape[-1]
    s, _ = token_scores(KB, QB)
    keep = residual_tokens(s, n_residual_tokens(T, ppm))
    Z = depth_factorize(KB)
    out = np.zeros(3)
    n_l, G, P, _ = QB.shape
    for m in MODES:
        if m == EXACT:
            continue
        Zk = np.zeros_like(Z)
        Zk[0] = Z[0]
        if m == RESIDUAL:
            Zk[1:, keep] = Z[1:, keep]
        Kh = depth_reconstruct(Zk)
        tot = 0.0
        for l in range(n_l):
            for g in range(G):
                Q = QB[l, g]
                tot += np.sum((Q @ Kh[l].T / math.sqrt(d) - Q @ KB[l].T / math.sqrt(d)) ** 2) / P
        out[m] = tot / (n_l * G)
    return out


def routing_errors_token_rates(KB, QB, rates_ppm) -> np.ndarray:
    """Eq. (2) for the shared mode and for the residual mode at every candidate
    fraction ``r_j`` of tokens: ``[E_S, E_R(r_0), ..., E_R(r_{J-1})]`` (E_E = 0).
    The paper chooses the fraction of each (block, head) by the routing loss
    budget (Section 3, after Eq. 2); here each fraction is one more candidate
    of the argmin of Eq. (3)."""
    out = [routing_errors_tokens(KB, QB, 0)[SHARED]]
    for r in rates_ppm:
        out.append(routing_errors_tokens(KB, QB, int(r))[RESIDUAL])
    return np.array(out)


def token_rate_candidates(d: int, rates_ppm, dtype: str, B: int = 2):
    """Omega of the candidates ``[shared, residual at r_0 .. r_{J-1}, exact]`` and the
    mode and fraction index of each (fraction index 0 for shared and exact)."""
    full = bytes_per_token_tokens(EXACT, d, 0, dtype, B)
    om = [bytes_per_token_tokens(SHARED, d, 0, dtype, B) / full]
    om += [bytes_per_token_tokens(RESIDUAL, d, int(r), dtype, B) / full for r in rates_ppm]
    om.append(1.0)
    modes = [SHARED] + [RESIDUAL] * len(rates_ppm) + [EXACT]
    idx = [0] + list(range(len(rates_ppm))) + [0]
    return np.array(om), modes, idx


def route_token_rates(E, T: int, d: int, rates_ppm, dtype: str, lam=None, budget=None, unit_sizes=None):
    """Routing with the residual fraction chosen per unit (Section 3: r_{b,h} by the
    routing loss budget): each unit takes the argmin of Eq. (3) over shared, exact and
    the residual mode at every candidate fraction, at ``lam``, or under the budget rule
    with ``budget`` bytes.  ``E``: ``[units][1 + J]`` from ``routing_errors_token_rates``.
    Returns ``(modes, rate_index, lambda, feasible)``."""
    E = np.asarray(E, dtype=np.float64)
    n, J = E.shape[0], len(rates_ppm)
    sizes = [2] * n if unit_sizes is None else [int(B) for B in unit_sizes]
    Ec = np.concatenate([E, np.zeros((n, 1))], axis=1)                  # exact costs nothing in Eq. 2
    cands = {B: token_rate_candidates(d, rates_ppm, dtype, B) for B in set(sizes)}
    om = np.stack([cands[B][0] for B in sizes])
    if budget is None:
        ch, lam_used, ok = route(Ec, om, lam), lam, True
    else:
        cb = np.array([[unit_bytes_tokens(cands[B][1][c], T, d, int(rates_ppm[cands[B][2][c]]) if c not in (0, J + 1)
                                          else 0, dtype, B) for c in range(J + 2)] for B in sizes])
        ch, lam_used, ok = route_budget_candidates(Ec, om, cb, budget)
    modes = np.array([cands[B][1][c] for B, c in zip(sizes, ch)], dtype=np.uint8)
    ridx = np.array([cands[B][2][c] for B, c in zip(sizes, ch)], dtype=np.uint8)
    return modes, ridx, lam_used, ok


_TOKEN_MASK_BYTES_PER_TOKEN = 1.0 / 8 + 4.0 / 128   # 1-bit token mask + a uint32 count per 128 tokens


def bytes_per_token_tokens(mode: int, d: int, ppm: int, dtype: str, B: int = 2) -> float:
    """Average bytes per token; residual heads pay r of the (B-1) high-frequency rows of K and V."""
    e, c = input_bytes(dtype), coef_bytes(dtype)
    if mode == RESIDUAL:
        return 2 * d * c + 2 * (B - 1) * d * c * (ppm / 1e6) + _TOKEN_MASK_BYTES_PER_TOKEN
    return float(bytes_per_token(mode, d, 0, dtype, B))


def omega_tokens(d: int, ppm: int, dtype: str, B: int = 2) -> np.ndarray:
    full = bytes_per_token_tokens(EXACT, d, ppm, dtype, B)
    return np.array([bytes_per_token_tokens(m, d, ppm, dtype, B) / full for m in MODES])


def unit_bytes_tokens(mode: int, T: int, d: int, ppm: int, dtype: str, B: int = 2) -> int:
    """Segment bytes with a token-level residual: M planes, the token mask
    (``ceil(T/32)`` uint32 words), the running count of residual tokens before
    every 128-token chunk (``ceil(T/128) + 1`` uint32), then the K and V
    high-frequency rows of the ``n`` residual tokens; every plane padded."""
    if mode != RESIDUAL:
        return unit_bytes(mode, T, d, 0, dtype, B)
    c = coef_bytes(dtype)
    n = n_residual_tokens(T, ppm)
    coef = _coef_plane(T, d, c)
    return (2 * coef + _plane(-(-T // 32) * 4) + _plane((-(-T // 128) + 1) * 4)
            + 2 * _plane(n * (B - 1) * d * c))


# ----------------------------------------------------------------------------
# generation: appended tokens and refreshed routing (Section 3, last
# paragraph of the method: one routing after prefill serves the whole
# decode, optionally re-decided at a fixed period of generated tokens)
# ----------------------------------------------------------------------------
def decode_spans(spans, tail_K, tail_V, layer: int, q, scale: float, d: int) -> np.ndarray:
    """Decode over a cache made of compressed spans followed by an exact tail.

    ``spans``: list of ``(unit, mode, B)`` for this (sequence, KV head), each
    a compressed stretch of consecutive tokens; ``tail_K``/``tail_V``:
    ``[n][d]`` exact rows of the generated tokens not yet compressed (n may
    be 0).  Attention runs over the concatenation of every span's
    reconstruction at ``layer`` and the tail: ``softmax(q K^T s) V``.
    """
    Ks, Vs = [], []
    for unit, mode, B in spans:
        pos = layer % B
        Ks.append(reconstruct_layer(unit, mode, pos, d, "K", B))
        Vs.append(reconstruct_layer(unit, mode, pos, d, "V", B))
    Ks.append(np.asarray(tail_K, dtype=np.float64).reshape(-1, d))
    Vs.append(np.asarray(tail_V, dtype=np.float64).reshape(-1, d))
    K = np.concatenate(Ks, axis=0)
    V = np.concatenate(Vs, axis=0)
    if K.shape[0] == 0:
        return np.zeros((np.asarray(q).shape[0], d))
    return attention(q, K, V, scale)


def refresh_modes(KB_tail, QB_recent, k: int, dtype: str, lam: float) -> int:
    """Mode of one (block, KV head) for a refreshed span: Eq. (2) on the span's
    own keys with the most recent decode queries as the probe rows, then the
    argmin of Eq. (3) at ``lam`` (the span's Omega follows its block size)."""
    E = routing_errors(KB_tail, QB_recent, k)
    B = np.asarray(KB_tail).shape[0]
    return int(route(E[None], omega(np.asarray(KB_tail).shape[-1], k, dtype, B), lam)[0])


# ----------------------------------------------------------------------------
# Eq. (2): routing loss
# ----------------------------------------------------------------------------
def candidate_keys(KB, mode: int, k: int) -> np.ndarray:
    """K^(m) of every layer of a block from unrounded coefficients, ``[B][T][d]``."""
    KB = np.asarray(KB, dtype=np.float64)
    B = KB.shape[0]
    if mode == EXACT:
        return KB.copy()
    Z = depth_factorize(KB)
    Zk = np.zeros_like(Z)
    Zk[0] = Z[0]
    if mode == RESIDUAL and k > 0:
        if B == 2:
            idx = residual_channels(KB[0], KB[1], k)
            np.put_along_axis(Zk[1], idx, np.take_along_axis(Z[1], idx, axis=-1), axis=-1)
        else:
            codes = residual_codes_dct4(KB, k)
            t = np.broadcast_to(np.arange(KB.shape[1])[:, None], codes.shape)
            Zk[codes & 3, t, codes >> 2] = Z[codes & 3, t, codes >> 2]
    return depth_reconstruct(Zk)


def routing_errors(KB, QB, k: int) -> np.ndarray:
    """Logit-reconstruction term of Eq. (2) for the three modes, ``[3]``.

    ``KB``: ``[B][T][d]`` keys of the block's layers for one KV head.
    ``QB``: ``[B][G][P][d]`` probe queries of those layers for the G query
    heads of the group.  The term is averaged over the B layers and the G
    heads: ``(1/(B G)) sum_{l,g} (1/P) sum_p ||q K^(m)T/sqrt(d) - q K^T/sqrt(d)||^2``.
    """
    KB = np.asarray(KB, dtype=np.float64)
    QB = np.asarray(QB, dtype=np.float64)
    d = KB.shape[-1]
    n_l, G, P, _ = QB.shape
    out = np.zeros(3, dtype=np.float64)
    for m in MODES:
        Kh = candidate_keys(KB, m, k)
        tot = 0.0
        for l in range(n_l):
            for g in range(G):
                Q = QB[l, g]
                exact_logits = Q @ KB[l].T / math.sqrt(d)
                recon_logits = Q @ Kh[l].T / math.sqrt(d)
                tot += np.sum((recon_logits - exact_logits) ** 2) / P
        out[m] = tot / (n_l * G)
    return out


# ----------------------------------------------------------------------------
# memory cost, layout bytes and routing
# ----------------------------------------------------------------------------
def _index_bytes(B: int) -> int:
    """Bytes of one residual index: a channel (B = 2) or a code 4 c + j (B = 4)."""
    return 1 if B == 2 else 2


def bytes_per_token(mode: int, d: int, k: int, dtype: str, B: int = 2) -> int:
    e, c = input_bytes(dtype), coef_bytes(dtype)
    if mode == SHARED:
        return 2 * d * c
    if mode == RESIDUAL:
        return 2 * d * c + 2 * k * (_index_bytes(B) + c)
    if mode == EXACT:
        return 2 * B * d * e
    raise ValueError(mode)


def omega(d: int, k: int, dtype: str, B: int = 2) -> np.ndarray:
    """Normalized memory cost Omega(m): bytes per token relative to exact mode."""
    full = bytes_per_token(EXACT, d, k, dtype, B)
    return np.array([bytes_per_token(m, d, k, dtype, B) / full for m in MODES], dtype=np.float64)


def _plane(nbytes: int) -> int:
    return -(-nbytes // PLANE_ALIGN) * PLANE_ALIGN


FP8_BLOCK = 1024


def _coef_plane(T: int, d: int, c: int) -> int:
    """A shared (M) plane: one-byte FP8 coefficients fill whole 1 KB blocks
    (a storage choice of the implementation, not of the paper: the decode
    reads two rows' pieces per 16-byte load), wider ones are padded to 256 B."""
    if c == 1:
        return _plane(-(-(T * d) // FP8_BLOCK) * FP8_BLOCK)
    return _plane(T * d * c)


def unit_bytes(mode: int, T: int, d: int, k: int, dtype: str, B: int = 2) -> int:
    """Bytes of one (sequence, block, KV head) segment; every plane padded to 256 B
    (FP8 shared planes to 1 KB)."""
    e, c = input_bytes(dtype), coef_bytes(dtype)
    coef = _coef_plane(T, d, c)
    if mode == SHARED:
        return 2 * coef
    if mode == RESIDUAL:
        return 2 * coef + 2 * (_plane(T * k * _index_bytes(B)) + _plane(T * k * c))
    if mode == EXACT:
        return 2 * B * _plane(T * d * e)
    raise ValueError(mode)


def cache_bytes(seq_lens, modes, d: int, k: int, dtype: str, sizes=None) -> int:
    """Total bytes of a cache; ``modes`` is ``[batch][blocks][Hkv]``, ``sizes`` the block sizes (pairs if None)."""
    modes = np.asarray(modes)
    if sizes is None:
        sizes = [2] * modes.shape[1]
    tot = 0
    for s, T in enumerate(seq_lens):
        for b, B in enumerate(sizes):
            for m in modes[s, b].reshape(-1):
                tot += unit_bytes(int(m), int(T), d, k, dtype, B)
    return tot


def _breakpoint(Ea: float, Eb: float, oa: float, ob: float) -> float:
    """The lambda at which mode a (the cheaper, ``oa < ob``) and mode b cost the same:
    ``Ea + lam oa = Eb + lam ob``."""
    return (Ea - Eb) / (ob - oa)


def _prefer(Ea: float, Eb: float, oa: float, ob: float, lam: float) -> bool:
    """Whether mode a wins against mode b at ``lam``, a being the cheaper one
    (``oa < ob``, or equal cost and the lower mode): a costs no more than b,
    ``Ea + lam oa <= Eb + lam ob``, i.e. ``lam >= breakpoint`` (ties go to the
    cheaper mode).  Deciding against the breakpoint itself, not against the two
    costs evaluated in floating point, makes a tie at a breakpoint exact: at
    ``lam`` equal to the breakpoint value the two costs are equal by definition,
    whereas ``Ea + lam oa`` and ``Eb + lam ob`` may round apart."""
    if oa == ob:
        return Ea <= Eb
    return lam >= _breakpoint(Ea, Eb, oa, ob)


def _cheaper_first(m1: int, m2: int, om) -> Tuple[int, int]:
    return (m1, m2) if (om[m1], m1) <= (om[m2], m2) else (m2, m1)


def route(E, om, lam: float) -> np.ndarray:
    """argmin_m E[u, m] + lam * Omega(m) (Eq. 3), ties to the cheaper mode.

    ``E`` is ``[units][C]`` and ``om`` is ``[C]`` or ``[units][C]``: C = 3 for the
    three modes, or more candidates (the residual mode at several fractions of
    tokens, ``route_token_rates``).  The candidates are compared in turn, each
    pair through ``_prefer``; the answer is a candidate index.
    """
    om = np.asarray(om, dtype=np.float64)
    C = om.shape[-1]
    E = np.asarray(E, dtype=np.float64).reshape(-1, C)
    om = np.broadcast_to(om, E.shape)
    out = np.zeros(E.shape[0], dtype=np.uint8)
    for u in range(E.shape[0]):
        best = 0
        for m in range(1, C):
            a, b = _cheaper_first(best, m, om[u])
            best = a if _prefer(E[u, a], E[u, b], om[u, a], om[u, b], lam) else b
        out[u] = best
    return out


def breakpoint_candidates(E, om) -> list:
    """Every positive finite breakpoint of every unit, between each pair of its candidates."""
    E = np.asarray(E, dtype=np.float64)
    om = np.broadcast_to(np.asarray(om, dtype=np.float64), E.shape)
    C = E.shape[-1]
    out = set()
    for u in range(E.shape[0]):
        for i in range(C):
            for j in range(i + 1, C):
                a, b = _cheaper_first(i, j, om[u])
                if not om[u, b] > om[u, a]:
                    continue
                lam = _breakpoint(E[u, a], E[u, b], om[u, a], om[u, b])
                if lam > 0 and np.isfinite(lam):
                    out.add(float(lam))
    return sorted(out)


def route_budget_candidates(E, om, cand_bytes, budget: int) -> Tuple[np.ndarray, float, bool]:
    """The budget rule over any candidate set: the smallest lambda among 0, every
    breakpoint and +inf whose footprint (the sum of each unit's chosen candidate's
    bytes, ``cand_bytes`` ``[units][C]``) is within ``budget``.  Returns
    ``(choices, lambda, feasible)``; infeasible gives each unit's cheapest candidate."""
    E = np.asarray(E, dtype=np.float64)
    om = np.broadcast_to(np.asarray(om, dtype=np.float64), E.shape)
    cand_bytes = np.asarray(cand_bytes)
    for lam in [0.0] + breakpoint_candidates(E, om) + [math.inf]:
        ch = route(E, om, lam)
        if sum(int(cand_bytes[u, c]) for u, c in enumerate(ch)) <= budget:
            return ch, lam, True
    return route(E, om, math.inf), math.inf, False


def route_budget(E, T: int, d: int, k: int, dtype: str, budget: int,
                 unit_sizes=None) -> Tuple[np.ndarray, float, bool]:
    """Smallest lambda (among 0, breakpoints, +inf) whose footprint fits ``budget``.

    ``E``: ``[units][3]``; ``unit_sizes``: the block size B of every unit
    (pairs if None).  Omega and the footprint of a unit follow its B.
    Returns ``(modes, lambda, feasible)``; when even all-shared exceeds the
    budget, returns all-shared and ``feasible=False``.
    """
    E = np.asarray(E, dtype=np.float64)
    n = E.shape[0]
    sizes = [2] * n if unit_sizes is None else [int(B) for B in unit_sizes]
    om = np.stack([omega(d, k, dtype, B) for B in sizes]) if n else np.zeros((0, 3))
    cands = {0.0}
    for u in range(n):
        for i in range(3):
            for j in range(i + 1, 3):
                a, b = _cheaper_first(i, j, om[u])
                if not om[u, b] > om[u, a]:
                    continue
                lam = _breakpoint(E[u, a], E[u, b], om[u, a], om[u, b])
                if lam > 0 and np.isfinite(lam):
                    cands.add(float(lam))
    order = sorted(cands) + [math.inf]
    seg = {(m, B): unit_bytes(m, T, d, k, dtype, B) for m in MODES for B in set(sizes)}
    for lam in order:
        modes = route(E, om, lam)
        fp = sum(seg[(int(m), B)] for m, B in zip(modes, sizes))
        if fp <= budget:
            return modes, lam, True
    return np.zeros(n, dtype=np.uint8), math.inf, False
