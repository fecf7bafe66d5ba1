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
  Eq. 3), a full softmax with max subtraction.

Readings of the paper adopted here (the paper leaves these open):

* blocks are adjacent layer pairs (B = 2) and ``F_2`` is the orthonormal
  DCT-II, i.e. the Haar matrix ``[[1, 1], [1, -1]] / sqrt(2)``;
* the residual keeps, for every token, the ``k`` channels of largest
  ``|x[2b] - x[2b+1]|`` (computed in float32 on the stored inputs; ties go to
  the lower channel; indices stored ascending), K and V chosen independently;
* what is stored is the per-layer image of each coefficient, ``P_k X`` with
  the projector ``P_k = F[k]^T F[k]``: ``M`` (the pair mean) for k = 0 and
  ``D`` (half the difference) for k = 1, so layer 2b reconstructs ``M + D``
  and layer 2b+1 ``M - D``; the projector entries are evaluated in 50-digit
  decimal arithmetic so that stored values are correctly rounded;
* the routing loss of a (pair, KV head) averages Eq. (2) over both layers of
  the pair and over the query heads of the KV head's group, uses the
  unrounded coefficients (storage rounding is not part of the method), and
  leaves values to follow the keys' decision;
* ``Omega(m)`` is the bytes per token of mode ``m`` divided by those of exact
  mode; ties in the argmin go to the cheaper mode;
* the budget rule takes the smallest ``lambda`` among 0, the per-head
  breakpoints and +inf whose footprint fits the budget;
* decode scales logits by ``1/sqrt(d)`` and attends over the cached tokens;
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
    ``s_k = sqrt(2/B)``.  The mirror symmetry ``F[k, B-1-n] = (-1)^k F[k, n]``
    of the DCT-II is applied exactly, so identical layers have exactly zero
    high-frequency coefficients.
    """
    F = np.empty((B, B), dtype=np.float64)
    for k in range(B):
        s = math.sqrt(1.0 / B) if k == 0 else math.sqrt(2.0 / B)
        for n in range((B + 1) // 2):
            F[k, n] = s * math.cos(math.pi * (2 * n + 1) * k / (2 * B))
            F[k, B - 1 - n] = F[k, n] if k % 2 == 0 else -F[k, n]
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
    """Z = F_B X along the leading (layer) axis of a block."""
    X = np.asarray(X, dtype=np.float64)
    F = dct_matrix(X.shape[0])
    Z = np.zeros_like(X)
    for k in range(X.shape[0]):
        for n in range(X.shape[0]):
            Z[k] += F[k, n] * X[n]
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


# ----------------------------------------------------------------------------
# Eq. (3): compressed representation of one (pair, KV head) unit
# ----------------------------------------------------------------------------
def compress_unit(K2, V2, mode: int, k: int, dtype: str) -> Dict[str, np.ndarray]:
    """Stored planes of one unit.

    ``K2, V2``: ``[2][T][d]`` inputs of layers 2b and 2b+1.  Returns a dict
    with ``MK, MV`` ([T][d]) for shared/residual heads, plus ``IK, VK, IV,
    VV`` ([T][k] indices and half-difference values) for residual heads, or
    ``K0, K1, V0, V1`` (the inputs) for exact heads.  Values are rounded to
    the storage precision.
    """
    out: Dict[str, np.ndarray] = {}
    if mode == EXACT:
        for name, X in (("K", K2), ("V", V2)):
            X = np.asarray(X, dtype=np.float64)
            out[name + "0"] = round_input(X[0], dtype)
            out[name + "1"] = round_input(X[1], dtype)
        return out
    for name, X in (("K", K2), ("V", V2)):
        X = np.asarray(X, dtype=np.float64)
        out["M" + name] = round_coef(coefficient_image(X, 0, 0), dtype)
        if mode == RESIDUAL:
            idx = residual_channels(X[0], X[1], k)
            D = coefficient_image(X, 1, 0)
            out["I" + name] = idx
            out["V" + name] = round_coef(np.take_along_axis(D, idx, axis=-1), dtype)
    return out


def reconstruct_layer(unit: Dict[str, np.ndarray], mode: int, parity: int, d: int, which: str) -> np.ndarray:
    """K~ or V~ (``which`` = "K"/"V") of layer 2b+parity from the stored planes (Eq. 3)."""
    if mode == EXACT:
        return np.asarray(unit[which + str(parity)], dtype=np.float64)
    F = dct_matrix(2)
    M = np.asarray(unit["M" + which], dtype=np.float64)
    T = M.shape[0]
    Z = np.zeros((2, T, d), dtype=np.float64)
    Z[0] = M / F[0, 0]
    if mode == RESIDUAL and unit["I" + which].shape[-1] > 0:
        idx = unit["I" + which]
        vals = np.asarray(unit["V" + which], dtype=np.float64) / F[1, 0]
        np.put_along_axis(Z[1], idx, vals, axis=-1)
    return depth_reconstruct(Z)[parity]


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


def decode_unit(unit, mode: int, layer: int, q, scale: float, d: int) -> np.ndarray:
    """Output rows ``[G][d]`` of the G query heads of one KV head at ``layer``."""
    parity = layer % 2
    Kt = reconstruct_layer(unit, mode, parity, d, "K")
    Vt = reconstruct_layer(unit, mode, parity, d, "V")
    return attention(q, Kt, Vt, scale)


# ----------------------------------------------------------------------------
# Eq. (2): routing loss
# ----------------------------------------------------------------------------
def candidate_keys(K2, mode: int, k: int) -> np.ndarray:
    """K^(m) of both layers of a pair from unrounded coefficients, ``[2][T][d]``."""
    K2 = np.asarray(K2, dtype=np.float64)
    if mode == EXACT:
        return K2.copy()
    Z = depth_factorize(K2)
    Zk = np.zeros_like(Z)
    Zk[0] = Z[0]
    if mode == RESIDUAL and k > 0:
        idx = residual_channels(K2[0], K2[1], k)
        np.put_along_axis(Zk[1], idx, np.take_along_axis(Z[1], idx, axis=-1), axis=-1)
    return depth_reconstruct(Zk)


def routing_errors(K2, Q2, k: int) -> np.ndarray:
    """Logit-reconstruction term of Eq. (2) for the three modes, ``[3]``.

    ``K2``: ``[2][T][d]`` keys of the pair's two layers for one KV head.
    ``Q2``: ``[2][G][P][d]`` probe queries of those layers for the G query
    heads of the group.  The term is averaged over the two layers and the G
    heads: ``(1/(2G)) sum_{l,g} (1/P) sum_p ||q K^(m)T/sqrt(d) - q K^T/sqrt(d)||^2``.
    """
    K2 = np.asarray(K2, dtype=np.float64)
    Q2 = np.asarray(Q2, dtype=np.float64)
    d = K2.shape[-1]
    n_l, G, P, _ = Q2.shape
    out = np.zeros(3, dtype=np.float64)
    for m in MODES:
        Kh = candidate_keys(K2, m, k)
        tot = 0.0
        for l in range(n_l):
            for g in range(G):
                Q = Q2[l, g]
                exact_logits = Q @ K2[l].T / math.sqrt(d)
                recon_logits = Q @ Kh[l].T / math.sqrt(d)
                tot += np.sum((recon_logits - exact_logits) ** 2) / P
        out[m] = tot / (n_l * G)
    return out


# ----------------------------------------------------------------------------
# memory cost, layout bytes and routing
# ----------------------------------------------------------------------------
def bytes_per_token(mode: int, d: int, k: int, dtype: str) -> int:
    e, c = input_bytes(dtype), coef_bytes(dtype)
    if mode == SHARED:
        return 2 * d * c
    if mode == RESIDUAL:
        return 2 * d * c + 2 * k * (1 + c)
    if mode == EXACT:
        return 4 * d * e
    raise ValueError(mode)


def omega(d: int, k: int, dtype: str) -> np.ndarray:
    """Normalized memory cost Omega(m): bytes per token relative to exact mode."""
    full = bytes_per_token(EXACT, d, k, dtype)
    return np.array([bytes_per_token(m, d, k, dtype) / full for m in MODES], dtype=np.float64)


def _plane(nbytes: int) -> int:
    return -(-nbytes // PLANE_ALIGN) * PLANE_ALIGN


def unit_bytes(mode: int, T: int, d: int, k: int, dtype: str) -> int:
    """Bytes of one (sequence, pair, KV head) segment; every plane padded to 256 B."""
    e, c = input_bytes(dtype), coef_bytes(dtype)
    coef = _plane(T * d * c)
    if mode == SHARED:
        return 2 * coef
    if mode == RESIDUAL:
        return 2 * coef + 2 * (_plane(T * k) + _plane(T * k * c))
    if mode == EXACT:
        return 4 * _plane(T * d * e)
    raise ValueError(mode)


def cache_bytes(seq_lens, modes, d: int, k: int, dtype: str) -> int:
    """Total bytes of a cache; ``modes`` is ``[batch][pairs][Hkv]``."""
    modes = np.asarray(modes)
    tot = 0
    for s, T in enumerate(seq_lens):
        for m in modes[s].reshape(-1):
            tot += unit_bytes(int(m), int(T), d, k, dtype)
    return tot


def route(E, om, lam: float) -> np.ndarray:
    """argmin_m E[u, m] + lam * Omega(m), ties to the cheaper (lower) mode."""
    E = np.asarray(E, dtype=np.float64)
    cost = E + lam * np.asarray(om, dtype=np.float64)
    if np.isinf(lam):
        cost = np.where(np.isnan(cost), np.inf, cost)
    return np.argmin(cost, axis=-1).astype(np.uint8)


def route_budget(E, T: int, d: int, k: int, dtype: str, budget: int) -> Tuple[np.ndarray, float, bool]:
    """Smallest lambda (among 0, breakpoints, +inf) whose footprint fits ``budget``.

    ``E``: ``[units][3]``.  Returns ``(modes, lambda, feasible)``; when even
    all-shared exceeds the budget, returns all-shared and ``feasible=False``.
    """
    E = np.asarray(E, dtype=np.float64)
    om = omega(d, k, dtype)
    cands = {0.0}
    for u in range(E.shape[0]):
        for i in range(3):
            for j in range(i + 1, 3):
                if not om[j] > om[i]:
                    continue
                lam = (E[u, i] - E[u, j]) / (om[j] - om[i])
                if lam > 0 and np.isfinite(lam):
                    cands.add(float(lam))
    order = sorted(cands) + [math.inf]
    seg = {m: unit_bytes(m, T, d, k, dtype) for m in MODES}
    for lam in order:
        modes = route(E, om, lam)
        fp = sum(seg[int(m)] for m in modes)
        if fp <= budget:
            return modes, lam, True
    return np.zeros(E.shape[0], dtype=np.uint8), math.inf, False
