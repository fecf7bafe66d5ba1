"""Parity of the HIP path (through the C ABI) with the CPU oracle.

Bars: residual channel indices, head modes and exact-mode planes bit-exact;
stored M/D values within 1 ulp of the storage type (the oracle rounds its
float64 DCT coefficients, the kernels round exact fp32 sums); attention
outputs within relative L2 error 1e-5 (fp32) / 1e-2 (bf16) per (sequence,
layer, query head); routing losses within 2e-5 relative: the MFMA Gram
takes each half difference as a bf16 hi + lo pair (its representation error is
2^-18 relative, the dropped lo lo^T term as small), so E carries a few 1e-6.
Head modes are compared at penalties between the oracle's breakpoints and
under the budget rule; a unit whose oracle cost margin is below 1e-4 would be
a near-tie, which the seeded cases must not contain.
"""
import math
import sys

import numpy as np
import pytest

import oracle as O
from synth import WORKLOADS, gen, scaled

from gpu_cases import (budget_defining_units, check_modes, compare_units, oracle_decode_layer, rel_l2,
                       separated_lambdas, sharpened_queries, unpack_unit)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2607_06519_amd import binding
    binding.load()          # a missing library must fail here, loudly
    return torch


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _upload(w, K, V):
    from paper_2607_06519_amd.cache import to_device
    Kd = to_device(K, w.dtype)
    Vd = to_device(V, w.dtype)
    return Kd, Vd, [Kd[l] for l in range(w.n_layers)], [Vd[l] for l in range(w.n_layers)]


def _run_compress(w, modes_b, Ks, Vs):
    """GPU compress of every sequence; returns (cache, per-seq device layer lists)."""
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import CompressedCache
    dm = B.dims(**w.dims())
    cache = CompressedCache(dm, w.seq_lens, modes_b)
    if w.dtype == "bf16_e4m3":
        cache.buf.fill_(0x7F)   # an E4M3 NaN in every byte compress leaves alone: decode must read none
    keep = []
    for s in range(w.batch):
        Kd, Vd, kl, vl = _upload(w, Ks[s], Vs[s])
        keep.append((Kd, Vd))
        cache.compress(s, kl, vl)
    return cache, keep


def _oracle_units(w, K, V, modes):
    return {(b, h): O.compress_unit(K[f:f + B, h], V[f:f + B, h], int(modes[b, h]), w.topk, w.dtype)
            for b, (f, B) in enumerate(w.blocks) for h in range(w.n_kv_heads)}


def _check_compress(w, cache, s, ref_units, K=None, V=None):
    buf = cache.host_bytes()
    T = w.seq_lens[s]
    nz = {}
    for (b, h), ref in ref_units.items():
        f, B = w.blocks[b]
        got = unpack_unit(buf, int(cache.offsets_host[s, b, h]), int(cache.modes_host[s, b, h]), T,
                          w.head_dim, w.topk, w.dtype, B)
        inputs = (K[f:f + B, h], V[f:f + B, h]) if (B == 4 and K is not None) else None
        st = compare_units(got, ref, w.dtype, inputs=inputs)
        for k_, v_ in st.items():
            nz[k_] = nz.get(k_, 0) + v_
    return nz


CASES = {
    "tiny": WORKLOADS["tiny"],
    "bf16_ragged": scaled(WORKLOADS["llama8b"], n_layers=4, seq_lens=(1000,), n_needles=6),
    "bf16_d64_k5": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=4, head_dim=64, topk=5,
                          seq_lens=(333,), n_needles=3, needle_channels=5),
    "f32_d128_k128": scaled(WORKLOADS["tiny"], head_dim=128, topk=128, n_q_heads=8, seq_lens=(200,),
                            needle_channels=8, fixed_modes=(1, 1, 0, 2)),
    "bf16_g8": scaled(WORKLOADS["long70b"], n_layers=2, n_kv_heads=2, n_q_heads=16, seq_lens=(777,), n_needles=4),
    "bf16_k0": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=4, topk=0, seq_lens=(300,),
                      n_needles=2, fixed_modes=(1, 0)),
    # FP8 E4M3 coefficients (bf16 inputs and exact heads)
    "e4m3_ragged": scaled(WORKLOADS["llama8b"], n_layers=4, seq_lens=(1000,), n_needles=6, dtype="bf16_e4m3"),
    "e4m3_d64_k8_g8": scaled(WORKLOADS["long70b"], n_layers=2, n_kv_heads=2, n_q_heads=16, head_dim=64, topk=8,
                             seq_lens=(517,), n_needles=3, needle_channels=8, dtype="bf16_e4m3"),
    "e4m3_k5": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=4, topk=5, seq_lens=(333,),
                      n_needles=3, needle_channels=5, dtype="bf16_e4m3"),
    # blocks of four layers (DCT-II(4)): all fours, and the mixed setting (pairs at both ends)
    "quads_bf16": scaled(WORKLOADS["llama8b"], n_layers=4, n_kv_heads=2, n_q_heads=8, seq_lens=(1000,),
                         n_needles=6, schedule=2, fixed_modes=(1, 1)),
    "mixed_bf16_l12": scaled(WORKLOADS["llama8b"], n_layers=12, n_kv_heads=2, n_q_heads=8, seq_lens=(777,),
                             n_needles=4, schedule=1, fixed_modes=(0, 1, 2, 1, 1, 2, 0, 1, 1, 0)),
    "quads_f32_d64_k7": scaled(WORKLOADS["tiny"], n_layers=4, n_kv_heads=2, n_q_heads=4, topk=7, seq_lens=(300,),
                               needle_channels=7, schedule=2, fixed_modes=(1, 2)),
    "quads_e4m3_g8": scaled(WORKLOADS["long70b"], n_layers=4, n_kv_heads=2, n_q_heads=16, seq_lens=(517,),
                            n_needles=3, dtype="bf16_e4m3", schedule=2, fixed_modes=(1, 0)),
    "quads_bf16_d64_k8": scaled(WORKLOADS["llama8b"], n_layers=4, n_kv_heads=2, n_q_heads=4, head_dim=64, topk=8,
                                seq_lens=(450,), n_needles=3, needle_channels=8, schedule=2, fixed_modes=(1, 1)),
    "quads_bf16_k40": scaled(WORKLOADS["llama8b"], n_layers=4, n_kv_heads=2, n_q_heads=4, topk=40,
                             seq_lens=(260,), n_needles=2, schedule=2, fixed_modes=(1, 2)),
    # the remaining shapes of the decode's reduce-scatter softmax: rows of 8 lanes (d = 64) with G = 4
    # (one logit per lane) and G = 1 (two butterfly stages), rows of 16 lanes with G = 1
    "bf16_d64_g4": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=8, head_dim=64, topk=8,
                          seq_lens=(600,), n_needles=3, needle_channels=8, fixed_modes=(1, 0)),
    "e4m3_d64_g1": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=2, head_dim=64, topk=8,
                          seq_lens=(530,), n_needles=3, needle_channels=8, dtype="bf16_e4m3", fixed_modes=(1, 2)),
    "bf16_g1": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=2, seq_lens=(520,), n_needles=3,
                      fixed_modes=(1, 0)),
}


def _modes(w, s=0):
    if w.fixed_modes is not None or w.mode_counts is not None:
        return gen.fixed_modes(w, s)
    raise ValueError


@pytest.mark.parametrize("name", list(CASES))
def test_compress_and_decode_parity(torch_dev, name):
    w = CASES[name]
    log(f"[case] compress+decode {name} T={w.seq_lens} d={w.head_dim} k={w.topk} {w.dtype}")
    K, V = gen.layer_cache(w, 0)
    modes = _modes(w)
    if name != "bf16_k0" and w.fixed_modes is None:
        # make sure all three modes appear
        modes = modes.copy()
        n = min(3, modes.size)
        modes.ravel()[:n] = [1, 2, 0][:n]
    cache, keep = _run_compress(w, modes[None], [K], [V])
    torch_dev.cuda.synchronize()
    ref = _oracle_units(w, K, V, modes)
    nz = _check_compress(w, cache, 0, ref, K, V)
    log(f"  compress ok; values 1 ulp apart: {nz}")
    tol = 1e-5 if w.dtype == "f32" else 1e-2
    worst = 0.0
    from paper_2607_06519_amd.cache import to_device
    for qi, qs in enumerate(sharpened_queries(w, 0, K)):
        for layer in range(w.n_layers):
            q = to_device(qs[layer], w.dtype)            # [batch=1][Hq][d]
            out = cache.decode(layer, q).float().cpu().numpy()[0]
            want = oracle_decode_layer(ref, modes, layer, qs[layer][0].astype(np.float64), w)
            for hq in range(w.n_q_heads):
                e = rel_l2(out[hq], want[hq])
                worst = max(worst, e)
                assert e <= tol, (name, qi, layer, hq, e)
    log(f"  decode ok; worst rel-L2 {worst:.3e} (tol {tol})")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_ragged_batch_decode(torch_dev, dtype):
    """Sequences of 1 to 1000 tokens and an empty one in one call: workgroups past a sequence's
    end leave empty records, which the merge skips; the empty sequence gets o = 0."""
    base = scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=8, n_needles=2, dtype=dtype)
    lens = (1, 100, 513, 1000, 0, 64)
    w = scaled(base, seq_lens=lens)
    tol = 1e-2 if dtype == "bf16" else 1e-5
    log(f"[case] ragged batch {lens} {dtype}")
    Ks, Vs, ref_units, modes_b = [], [], [], []
    for s, T in enumerate(lens):
        ws_ = scaled(base, seq_lens=(max(T, 1),))
        K, V = gen.layer_cache(ws_, 0)
        K, V = K[:, :, :T], V[:, :, :T]
        m = np.array([[s % 3, (s + 1) % 3]], np.uint8)
        Ks.append(K)
        Vs.append(V)
        modes_b.append(m)
        ref_units.append(_oracle_units(scaled(base, seq_lens=(T,)), K, V, m) if T > 0 else None)
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import CompressedCache, to_device
    cache = CompressedCache(B.dims(**w.dims()), lens, np.stack(modes_b))
    keep = []
    for s, T in enumerate(lens):
        if T == 0:
            continue
        Kd, Vd, kl, vl = _upload(scaled(base, seq_lens=(T,)), Ks[s], Vs[s])
        keep.append((Kd, Vd))
        cache.compress(s, kl, vl)
    qs = gen.decode_queries(w, 1, scale=8.0)
    for layer in range(2):
        q = to_device(qs[layer], w.dtype)
        out = cache.decode(layer, q).float().cpu().numpy()
        for s, T in enumerate(lens):
            if T == 0:
                assert np.all(out[s] == 0.0)
                continue
            want = oracle_decode_layer(ref_units[s], modes_b[s], layer, qs[layer][s].astype(np.float64),
                                       scaled(base, seq_lens=(T,)))
            for hq in range(w.n_q_heads):
                assert rel_l2(out[s, hq], want[hq]) <= tol, (s, layer, hq)
    log("  ragged ok")


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_all_empty_decode(torch_dev, dtype):
    """A call in which every sequence is empty (max_seq_len 0) writes o = 0, and a later call on
    the same workspace is unaffected."""
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import CompressedCache, to_device
    base = scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=8, n_needles=2, dtype=dtype)
    log(f"[case] all-empty batch {dtype}")
    w0 = scaled(base, seq_lens=(0, 0))
    cache = CompressedCache(B.dims(**w0.dims()), (0, 0), np.zeros((2, 1, 2), np.uint8))
    qs = gen.decode_queries(w0, 0, scale=8.0)
    for layer in range(2):
        q = to_device(qs[layer], w0.dtype)
        out = torch_dev.full_like(q, 7.0)
        cache.decode(layer, q, out)
        assert np.all(out.float().cpu().numpy() == 0.0), layer
    w1 = scaled(base, seq_lens=(300,))
    K, V = gen.layer_cache(w1, 0)
    modes = np.array([[1, 2]], np.uint8)
    ref = _oracle_units(w1, K, V, modes)
    Kd, Vd, kl, vl = _upload(w1, K, V)
    cache1 = CompressedCache(B.dims(**w1.dims()), (300,), modes[None])
    cache1.ws = cache.ws if cache.ws.numel() >= cache1.ws.numel() else cache1.ws
    cache1.compress(0, kl, vl)
    qs1 = gen.decode_queries(w1, 0, scale=8.0)
    for layer in range(2):
        out = cache1.decode(layer, to_device(qs1[layer], w1.dtype)).float().cpu().numpy()[0]
        want = oracle_decode_layer(ref, modes, layer, qs1[layer][0].astype(np.float64), w1)
        for hq in range(w1.n_q_heads):
            assert rel_l2(out[hq], want[hq]) <= (1e-2 if dtype == "bf16" else 1e-5), (layer, hq)
    log("  all-empty ok")


PROBE_CASES = {
    "tiny": WORKLOADS["tiny"],
    "bf16_small": scaled(WORKLOADS["prefill8b"], n_layers=4, n_kv_heads=4, n_q_heads=16, seq_lens=(1500,), n_probe=48),
    "bf16_g1_d64": scaled(WORKLOADS["prefill8b"], n_layers=2, n_kv_heads=3, n_q_heads=3, head_dim=64, topk=7,
                          seq_lens=(700,), n_probe=20, needle_channels=7),
    "quads_bf16": scaled(WORKLOADS["prefill8b"], n_layers=4, n_kv_heads=2, n_q_heads=8, seq_lens=(1500,), n_probe=48,
                         schedule=2),
    "mixed_bf16_d64_k7": scaled(WORKLOADS["prefill8b"], n_layers=12, n_kv_heads=2, n_q_heads=4, head_dim=64, topk=7,
                                seq_lens=(700,), n_probe=20, needle_channels=7, schedule=1),
    "quads_f32": scaled(WORKLOADS["tiny"], n_layers=4, n_kv_heads=2, n_q_heads=4, seq_lens=(600,), n_probe=24,
                        schedule=2),
    "f32_d128": scaled(WORKLOADS["tiny"], n_layers=2, n_kv_heads=2, n_q_heads=4, head_dim=128, topk=16,
                       seq_lens=(700,), n_probe=16, needle_channels=16),
}


@pytest.mark.parametrize("name", list(PROBE_CASES))
def test_probe_parity(torch_dev, name):
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import probe, to_device
    w = PROBE_CASES[name]
    log(f"[case] probe {name}")
    K, _ = gen.layer_cache(w, 0)
    Q = gen.probe_queries(w, 0)
    Kd = to_device(K, w.dtype)
    Qd = to_device(Q, w.dtype)
    dm = B.dims(**w.dims())
    err, ws = probe(dm, w.seq_lens[0], [Kd[l] for l in range(w.n_layers)], [Qd[l] for l in range(w.n_layers)],
                    w.n_probe)
    got = err.cpu().numpy().astype(np.float64)
    G = w.group
    ref = np.zeros((w.n_blocks, w.n_kv_heads, 3))
    for b, (f, Bs) in enumerate(w.blocks):
        for h in range(w.n_kv_heads):
            ref[b, h] = O.routing_errors(K[f:f + Bs, h], Q[f:f + Bs, h * G:(h + 1) * G], w.topk)
    relerr = np.abs(got - ref[..., :2]) / np.abs(ref[..., :2])
    log(f"  max rel error of E: {relerr.max():.3e}")
    assert relerr.max() <= 2e-5
    # modes at penalties between the oracle's breakpoints, then under the budget rule
    om = np.stack([O.omega(w.head_dim, w.topk, w.dtype, Bs) for Bs in w.block_sizes for _ in range(w.n_kv_heads)])
    E3 = ref.reshape(-1, 3)
    for lam in separated_lambdas(E3, om):
        gm, _, _ = B.route(dm, w.seq_lens[0], got.astype(np.float32), lam=float(lam))
        check_modes(gm, E3, om, lam, name)
    T = w.seq_lens[0]
    seg = {(m, Bs): O.unit_bytes(m, T, w.head_dim, w.topk, w.dtype, Bs) for m in O.MODES for Bs in (2, 4)}
    sizes = [Bs for Bs in w.block_sizes for _ in range(w.n_kv_heads)]
    lo = sum(seg[(0, Bs)] for Bs in sizes)
    hi = sum(seg[(2, Bs)] for Bs in sizes)
    for frac in (0.3, 0.7):
        budget = int(lo + frac * (hi - lo))
        want_m, want_lam, ok = O.route_budget(E3, T, w.head_dim, w.topk, w.dtype, budget, sizes)
        gm, glam, st = B.route(dm, T, got.astype(np.float32), budget_bytes=budget)
        assert ok and st == 0
        tied = budget_defining_units(E3, om, want_lam)
        assert abs(glam / want_lam - 1.0) <= 1e-4, (glam, want_lam)
        # the GPU's lambda* is the breakpoint of the same unit(s), computed from its own losses
        gE3 = np.concatenate([got.reshape(-1, 2).astype(np.float32).astype(np.float64),
                              np.zeros((len(E3), 1))], axis=1)
        assert budget_defining_units(gE3, om, glam) == tied, (tied, budget_defining_units(gE3, om, glam))
        check_modes(gm, E3, om, want_lam, f"{name} budget {frac}", exclude=tied)
        np.testing.assert_array_equal(gm.ravel()[tied], want_m[tied])


TIE_CASES = {
    # rows on LPR = 16 lanes (bf16, d = 128), k below and above LPR, k = d
    "bf16_k8": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=4, topk=8, seq_lens=(515,),
                      n_needles=0, fixed_modes=(1, 1)),
    "bf16_k40": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=4, topk=40, seq_lens=(131,),
                       n_needles=0, fixed_modes=(1, 1)),
    "bf16_k128": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=1, n_q_heads=2, topk=128, seq_lens=(70,),
                        n_needles=0, fixed_modes=(1,)),
    # 32 lanes (f32, d = 128), 8 lanes (bf16, d = 64), FP8 values
    "f32_k16": scaled(WORKLOADS["tiny"], n_layers=2, n_kv_heads=2, n_q_heads=4, head_dim=128, topk=16,
                      seq_lens=(203,), n_needles=0, fixed_modes=(1, 1)),
    "f32_d64_k7": scaled(WORKLOADS["tiny"], n_layers=2, n_kv_heads=2, n_q_heads=4, head_dim=64, topk=7,
                         seq_lens=(97,), n_needles=0, fixed_modes=(1, 1)),
    "bf16_d64_k5": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=4, head_dim=64, topk=5,
                          seq_lens=(333,), n_needles=0, fixed_modes=(1, 1)),
    "e4m3_k12": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=4, topk=12, seq_lens=(300,),
                       n_needles=0, fixed_modes=(1, 1), dtype="bf16_e4m3"),
    "bf16_k1": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=1, n_q_heads=2, topk=1, seq_lens=(129,),
                      n_needles=0, fixed_modes=(1,)),
    # blocks of four: 3d coefficients per row, 24 keys a lane (bf16) or 12 (fp32)
    "quads_bf16_k16": scaled(WORKLOADS["llama8b"], n_layers=4, n_kv_heads=2, n_q_heads=4, topk=16, seq_lens=(301,),
                             n_needles=0, schedule=2, fixed_modes=(1, 1)),
    "quads_bf16_k1": scaled(WORKLOADS["llama8b"], n_layers=4, n_kv_heads=1, n_q_heads=2, topk=1, seq_lens=(77,),
                            n_needles=0, schedule=2, fixed_modes=(1,)),
    "quads_bf16_k128": scaled(WORKLOADS["llama8b"], n_layers=4, n_kv_heads=1, n_q_heads=2, topk=128, seq_lens=(65,),
                              n_needles=0, schedule=2, fixed_modes=(1,)),
    "quads_f32_d64_k7": scaled(WORKLOADS["tiny"], n_layers=4, n_kv_heads=2, n_q_heads=4, head_dim=64, topk=7,
                               seq_lens=(99,), n_needles=0, schedule=2, fixed_modes=(1, 1)),
}


def _tie_heavy(K, V, seed: int):
    """Inputs whose residual keys tie often: values on a coarse grid, every
    7th token with equal layers (all keys zero), every 11th with each later
    layer a constant shift of the first (pairs: all keys equal)."""
    rng = np.random.default_rng(seed)
    out = []
    for X in (K, V):
        X = np.round(X * 4.0) / 4.0
        X += rng.integers(-2, 3, size=X.shape) * 0.25 * (rng.random(X.shape) < 0.3)
        X = np.clip(X, -4.0, 4.0).astype(np.float32)
        T = X.shape[2]
        for n in range(1, X.shape[0]):
            X[n, :, 0:T:7] = X[0, :, 0:T:7]
            X[n, :, 0:T:11] = X[0, :, 0:T:11] + np.float32(0.5 * n)
        out.append(X)
    return out


@pytest.mark.parametrize("name", list(TIE_CASES))
def test_compress_residual_ties(torch_dev, name):
    """Residual entries under heavy ties: pairs' indices bit-exact (ties to the
    lower channel) with values within 1 ulp; blocks of four's codes by the
    near-tie rule of check_quad_codes (ties to the lower code) with values
    within the butterfly's bound."""
    w = TIE_CASES[name]
    log(f"[case] compress ties {name} T={w.seq_lens} d={w.head_dim} k={w.topk} {w.dtype}")
    K, V = gen.layer_cache(w, 0)
    K, V = _tie_heavy(K, V, 7 + len(name))
    modes = _modes(w)
    cache, keep = _run_compress(w, modes[None], [K], [V])
    torch_dev.cuda.synchronize()
    ref = _oracle_units(w, K, V, modes)
    nz = _check_compress(w, cache, 0, ref, K, V)
    log(f"  ties ok; values 1 ulp apart: {nz}")


REUSE_CASES = {
    "bf16_k16": scaled(WORKLOADS["llama8b"], n_layers=4, n_kv_heads=2, n_q_heads=8, seq_lens=(1000,), n_probe=16,
                       n_needles=4, fixed_modes=(1, 0, 1, 2)),
    "f32_d64_k7": scaled(WORKLOADS["tiny"], n_layers=2, n_kv_heads=2, n_q_heads=4, head_dim=64, topk=7,
                         seq_lens=(333,), n_probe=8, n_needles=0, fixed_modes=(1, 1)),
    # fp32 rows of 128: the probe ranks them on 8 lanes of four runs each
    "f32_k16": scaled(WORKLOADS["tiny"], n_layers=2, n_kv_heads=2, n_q_heads=4, head_dim=128, topk=16,
                      seq_lens=(290,), n_probe=8, n_needles=0, needle_channels=16, fixed_modes=(1, 1)),
    "e4m3_d64_k5": scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=4, head_dim=64, topk=5,
                          seq_lens=(517,), n_probe=8, n_needles=2, dtype="bf16_e4m3", fixed_modes=(1, 1)),
    "mixed_bf16": scaled(WORKLOADS["llama8b"], n_layers=12, n_kv_heads=2, n_q_heads=4, seq_lens=(300,), n_probe=8,
                         n_needles=2, schedule=1, fixed_modes=(1, 1, 0, 1, 1, 2, 1, 0, 1, 1)),
    "quads_f32_d64_k7": scaled(WORKLOADS["tiny"], n_layers=4, n_kv_heads=2, n_q_heads=4, head_dim=64, topk=7,
                               seq_lens=(211,), n_probe=8, n_needles=0, schedule=2, fixed_modes=(1, 1)),
    "quads_e4m3_k16": scaled(WORKLOADS["llama8b"], n_layers=4, n_kv_heads=2, n_q_heads=4, seq_lens=(260,), n_probe=8,
                             n_needles=2, schedule=2, dtype="bf16_e4m3", fixed_modes=(1, 1)),
}


@pytest.mark.parametrize("name", list(REUSE_CASES))
@pytest.mark.parametrize("ties", [False, True])
def test_compress_reuses_probe_selection(torch_dev, name, ties):
    """Compress taking the probe's K selections writes exactly the cache that
    compress selecting in its own pass writes (random and tie-heavy inputs)."""
    from paper_2607_06519_amd.cache import probe, to_device
    w = REUSE_CASES[name]
    log(f"[case] compress with the probe's selections {name} ties={ties}")
    K, V = gen.layer_cache(w, 0)
    if ties:
        for f in range(0, w.n_layers, 2):
            K[f:f + 2], V[f:f + 2] = _tie_heavy(K[f:f + 2], V[f:f + 2], 3 + f)
    Q = gen.probe_queries(w, 0)
    Kd, Vd, Qd = to_device(K, w.dtype), to_device(V, w.dtype), to_device(Q, w.dtype)
    kl, vl, ql = ([X[l] for l in range(w.n_layers)] for X in (Kd, Vd, Qd))
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import CompressedCache
    dm = B.dims(**w.dims())
    _, ksel = probe(dm, w.seq_lens[0], kl, ql, w.n_probe)
    modes = _modes(w)[None]
    a = CompressedCache(dm, w.seq_lens, modes)
    b = CompressedCache(dm, w.seq_lens, modes)
    a.buf.zero_()
    b.buf.zero_()
    a.compress(0, kl, vl)
    b.compress(0, kl, vl, k_select=ksel)
    torch_dev.cuda.synchronize()
    np.testing.assert_array_equal(a.host_bytes(), b.host_bytes())
    if ties:
        nz = _check_compress(w, b, 0, _oracle_units(w, K, V, _modes(w)), K, V)
        log(f"  equal to the oracle; values 1 ulp apart: {nz}")


def test_probe_deterministic(torch_dev):
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import probe, to_device
    w = PROBE_CASES["bf16_small"]
    K, _ = gen.layer_cache(w, 0)
    Q = gen.probe_queries(w, 0)
    Kd, Qd = to_device(K, w.dtype), to_device(Q, w.dtype)
    dm = B.dims(**w.dims())
    kl, ql = [Kd[l] for l in range(w.n_layers)], [Qd[l] for l in range(w.n_layers)]
    a, _ = probe(dm, w.seq_lens[0], kl, ql, w.n_probe)
    b, _ = probe(dm, w.seq_lens[0], kl, ql, w.n_probe)
    assert torch_dev.equal(a, b)


@pytest.mark.parametrize("dtype", ["bf16", "f32"])
def test_invalid_unit_gives_nan(torch_dev, dtype):
    """A unit whose mode is above exact or whose segment offset is not a multiple of 256
    is not read: its query heads' outputs come out NaN, every other head is unaffected."""
    torch = torch_dev
    from paper_2607_06519_amd.cache import to_device
    w = scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=4, n_q_heads=8, seq_lens=(600,), n_needles=2, dtype=dtype)
    K, V = gen.layer_cache(w, 0)
    modes = np.array([[0, 1, 2, 1]], np.uint8)
    cache, keep = _run_compress(w, modes[None], [K], [V])
    ref = _oracle_units(w, K, V, modes)
    q = gen.decode_queries(w, 0, scale=8.0)
    tol = 1e-5 if dtype == "f32" else 1e-2
    good_modes, good_offs = cache.modes.clone(), cache.offsets.clone()
    for bad in ("mode", "offset"):
        cache.modes.copy_(good_modes)
        cache.offsets.copy_(good_offs)
        if bad == "mode":
            cache.modes[0, 0, 1] = 3
        else:
            cache.offsets[0, 0, 2] += 16
        for layer in range(2):
            out = cache.decode(layer, to_device(q[layer], dtype)).float().cpu().numpy()[0]
            want = oracle_decode_layer(ref, modes, layer, q[layer][0].astype(np.float64), w)
            badh = 1 if bad == "mode" else 2
            for hq in range(w.n_q_heads):
                if hq // w.group == badh:
                    assert np.all(np.isnan(out[hq])), (bad, layer, hq)
                else:
                    assert rel_l2(out[hq], want[hq]) <= tol, (bad, layer, hq)
    cache.modes.copy_(good_modes)
    cache.offsets.copy_(good_offs)
    log("  invalid units give NaN, the other heads match the oracle")


def test_partial_and_combine(torch_dev):
    """fdkv_decode_partial followed by fdkv_decode_combine equals fdkv_decode_attn bit for bit;
    and a sequence split in two token ranges, each compressed on its own and run through the
    partial phase separately (as two devices would), combines from the concatenated records into
    the oracle's attention over the whole sequence (the sequence-split merge of the records)."""
    torch = torch_dev
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import CompressedCache, to_device
    w = scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=4, n_q_heads=16, seq_lens=(1300, 900), n_needles=3)
    H, G, d = w.n_kv_heads, w.group, w.head_dim
    scale = 1.0 / math.sqrt(d)
    modes = np.stack([gen.fixed_modes(w, s) for s in range(w.batch)])
    modes[:, 0, :3] = [0, 1, 2]
    Ks, Vs = [], []
    for s, T in enumerate(w.seq_lens):
        K, V = gen.layer_cache(scaled(w, seq_lens=(T,)), 0)
        Ks.append(K)
        Vs.append(V)
    whole, keep = _run_compress(w, modes, Ks, Vs)
    qs = gen.decode_queries(w, 2, scale=8.0)
    # the two phases against the one call
    for layer in range(2):
        q = to_device(qs[layer], w.dtype)
        want = whole.decode(layer, q).clone()
        ws = torch.zeros_like(whole.ws)
        B.decode_partial(whole.dims, whole.batch, whole.seq_lens, whole.max_seq_len, whole.modes, whole.offsets,
                         whole.buf, layer, q, scale, ws)
        got = torch.empty_like(want)
        B.decode_combine(whole.dims, whole.batch, -(-whole.max_seq_len // 512), got, ws)
        torch.cuda.synchronize()
        assert torch.equal(got, want), layer
    # a sequence split at token 700 / 500: two caches of the token ranges, records concatenated per head
    cut = (700, 500)
    parts = []
    for lo_hi in ((0, cut), (cut, None)):
        lens = tuple((c if lo_hi[0] == 0 else T - c) for T, c in zip(w.seq_lens, cut))
        sub = [(K[:, :, :c] if lo_hi[0] == 0 else K[:, :, c:], V[:, :, :c] if lo_hi[0] == 0 else V[:, :, c:])
               for K, V, c in zip(Ks, Vs, cut)]
        wp = scaled(w, seq_lens=lens)
        cache, kp = _run_compress(wp, modes, [a for a, _ in sub], [b for _, b in sub])
        parts.append((wp, cache, kp, sub))
    for layer in range(2):
        q = to_device(qs[layer], w.dtype)
        recs = []
        for wp, cache, _, _ in parts:
            n = -(-wp.max_seq_len // 512)
            ws = torch.zeros(w.batch * H * n * G * (d + 4), dtype=torch.float32, device="cuda")
            B.decode_partial(cache.dims, cache.batch, cache.seq_lens, cache.max_seq_len, cache.modes,
                             cache.offsets, cache.buf, layer, q, scale, ws)
            recs.append(ws.view(w.batch, H, n, G * (d + 4)))
        cat = torch.cat(recs, dim=2).contiguous()
        out = torch.empty((w.batch, w.n_q_heads, d), dtype=torch.bfloat16, device="cuda")
        B.decode_combine(B.dims(**w.dims()), w.batch, cat.shape[2], out, cat.view(-1))
        got = out.float().cpu().numpy()
        for s in range(w.batch):
            for h in range(H):
                spans = []
                for wp, _, _, sub in parts:
                    Kp, Vp = sub[s]
                    m = int(modes[s, 0, h])
                    spans.append((O.compress_unit(Kp[0:2, h], Vp[0:2, h], m, w.topk, w.dtype), m, 2))
                ref = O.decode_spans(spans, np.zeros((0, d)), np.zeros((0, d)), layer,
                                     qs[layer][s, h * G:(h + 1) * G].astype(np.float64), scale, d)
                for g in range(G):
                    e = rel_l2(got[s, h * G + g], ref[g])
                    assert e <= 1e-2, (layer, s, h, g, e)
    log("  partial + combine equal the one call; a sequence split in two ranges combines to the oracle")
