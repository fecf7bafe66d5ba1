"""Parity at the workloads' full per-layer sizes, on sampled units.

A decode launch depends on (T, KV heads, query heads, d, k, batch), not on
the number of layers, so one layer pair at the full context length runs the
exact launch configuration the benchmark times.  The GPU path runs on every
head; the oracle recomputes a sample of (sequence, pair, KV head) units one
by one: their stored planes (bit-exact indices, values within 1 ulp) and the
attention outputs of their query heads in both layers of the pair.
"""
import math
import sys

import numpy as np
import pytest

import oracle as O
from synth import WORKLOADS, gen, scaled

from gpu_cases import budget_defining_units, check_modes, compare_units, rel_l2, separated_lambdas, unpack_unit

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_mod():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2607_06519_amd import binding
    binding.load()
    return torch


def _build_cache(torch, w, modes_b):
    """Generate every segment of every sequence on the device and compress it."""
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import CompressedCache, torch_dtype
    tdt = torch_dtype(w.dtype)
    cache = CompressedCache(B.dims(**w.dims()), w.seq_lens, modes_b)
    for s in range(w.batch):
        T = w.seq_lens[s]
        Kd = torch.empty((w.n_layers, w.n_kv_heads, T, w.head_dim), dtype=tdt, device="cuda")
        Vd = torch.empty_like(Kd)
        for b, h, k, v in gen.iter_segments(w, s, threads=16):
            f, nb = w.blocks[b]
            Kd[f:f + nb, h].copy_(torch.from_numpy(k).cuda().to(tdt))
            Vd[f:f + nb, h].copy_(torch.from_numpy(v).cuda().to(tdt))
        cache.compress(s, [Kd[l] for l in range(w.n_layers)], [Vd[l] for l in range(w.n_layers)])
        torch.cuda.synchronize()
        del Kd, Vd
    return cache


def _check_units(torch, w, cache, modes_b, samples, qscale=8.0):
    from paper_2607_06519_amd.cache import to_device
    buf = cache.host_bytes()
    G, d = w.group, w.head_dim
    q = gen.decode_queries(w, 0, scale=qscale)              # [L][batch][Hq][d]
    outs = [cache.decode(layer, to_device(q[layer], w.dtype)).float().cpu().numpy() for layer in range(w.n_layers)]
    worst = 0.0
    for (s, b, h) in samples:
        T = w.seq_lens[s]
        mode = int(modes_b[s, b, h])
        K, V, _ = gen.block_segment(w, s, b, h)
        f, nb = w.blocks[b]
        ref = O.compress_unit(K, V, mode, w.topk, w.dtype)
        got = unpack_unit(buf, int(cache.offsets_host[s, b, h]), mode, T, d, w.topk, w.dtype, nb)
        compare_units(got, ref, w.dtype, inputs=(K, V) if nb == 4 else None)
        for layer in range(f, f + nb):
            qq = q[layer][s, h * G:(h + 1) * G].astype(np.float64)
            want = O.decode_unit(ref, mode, layer, qq, 1.0 / math.sqrt(d), d, nb)
            for g in range(G):
                e = rel_l2(outs[layer][s, h * G + g], want[g])
                worst = max(worst, e)
                assert e <= 1e-2, (s, b, h, layer, g, e)
        log(f"  unit seq={s} block={b} head={h} mode={mode} T={T} ok")
    return worst


def _samples_by_mode(modes_b, per_mode=1, seqs=None):
    out = []
    seqs = range(modes_b.shape[0]) if seqs is None else seqs
    for m in (O.SHARED, O.RESIDUAL, O.EXACT):
        n = 0
        for s in seqs:
            for b in range(modes_b.shape[1]):
                for h in range(modes_b.shape[2]):
                    if modes_b[s, b, h] == m and n < per_mode:
                        out.append((s, b, h))
                        n += 1
    return out


@pytest.mark.parametrize("name,per_mode", [("llama8b", 2), ("long70b", 1), ("llama8b_quads", 2), ("llama8b_e4m3", 2)])
def test_fullsize_single_sequence(torch_mod, name, per_mode):
    if name == "llama8b_quads":    # one block of four layers at the full 8B shape
        w = scaled(WORKLOADS["llama8b_mixed"], n_layers=4, schedule=2)
    else:
        w = scaled(WORKLOADS[name], n_layers=2)
    log(f"[case] full-size {name}: T={w.seq_lens[0]} Hkv={w.n_kv_heads} Hq={w.n_q_heads} k={w.topk}")
    modes = gen.fixed_modes(w)[None].copy()
    modes[0, 0, :3] = [0, 1, 2]
    cache = _build_cache(torch_mod, w, modes)
    worst = _check_units(torch_mod, w, cache, modes, _samples_by_mode(modes, per_mode))
    log(f"  worst rel-L2 {worst:.3e}")


def test_fullsize_ragged_batch(torch_mod):
    w = scaled(WORKLOADS["batched8b"], n_layers=2)
    log(f"[case] full-size batched8b: lens {w.seq_lens}")
    modes = np.stack([gen.fixed_modes(w, s) for s in range(w.batch)])
    for s in range(w.batch):
        modes[s, 0, :3] = np.roll([0, 1, 2], s)
    cache = _build_cache(torch_mod, w, modes)
    samples = [(s, 0, h) for s, h in ((0, 0), (3, 1), (7, 2), (11, 5), (15, 7))]
    worst = _check_units(torch_mod, w, cache, modes, samples)
    log(f"  worst rel-L2 {worst:.3e}")


@pytest.mark.parametrize("nl,sched", [(2, 0), (4, 2)])
def test_fullsize_probe(torch_mod, nl, sched):
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import probe, torch_dtype
    w = scaled(WORKLOADS["prefill8b"], n_layers=nl, schedule=sched)
    T, P, G = w.seq_lens[0], w.n_probe, w.group
    log(f"[case] full-size probe: T={T} P={P} G={G} block of {nl}")
    tdt = torch_dtype(w.dtype)
    Kd = torch_mod.empty((nl, w.n_kv_heads, T, w.head_dim), dtype=tdt, device="cuda")
    segs = {}
    for b, h, k, v in gen.iter_segments(w, 0, threads=16):
        Kd[:, h].copy_(torch_mod.from_numpy(k).cuda().to(tdt))
        segs[h] = k
    Q = gen.probe_queries(w, 0)
    Qd = torch_mod.from_numpy(Q).cuda().to(tdt)
    err, _ = probe(B.dims(**w.dims()), T, [Kd[l] for l in range(nl)], [Qd[l] for l in range(nl)], P)
    got = err.cpu().numpy()[0].astype(np.float64)
    worst = 0.0
    for h in range(w.n_kv_heads):
        ref = O.routing_errors(segs[h], Q[:, h * G:(h + 1) * G], w.topk)
        rel = np.abs(got[h] - ref[:2]) / ref[:2]
        worst = max(worst, rel.max())
        log(f"  head {h}: E_S {got[h, 0]:.8g} vs {ref[0]:.8g}, E_R {got[h, 1]:.8g} vs {ref[1]:.8g}, rel {rel.max():.2e}")
        assert rel.max() <= 2e-5
    log(f"  worst rel error of E {worst:.2e}")


def test_fullsize_prefill_routing(torch_mod):
    """The whole 8B prefill routing: fdkv_probe over all 32 layers (128 units, T = 32768,
    P = 256, G = 4) and the budget rule of fdkv_route with the byte budget of the seeded
    50/35/15 mix, against the oracle's literal Eq. 2 and budget search
    (tests/golden/prefill8b_routing.json, written by make_prefill8b_routing.py):
    every loss within 2e-5, lambda* the breakpoint of the same unit within 1e-4, and
    every mode bit-exact (no other unit within 1e-4 of a tie at lambda*)."""
    import json
    import os
    torch = torch_mod
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import probe, torch_dtype
    with open(os.path.join(os.path.dirname(__file__), "golden", "prefill8b_routing.json")) as f:
        gold = json.load(f)
    w = WORKLOADS["prefill8b"]
    T, P, L, H, d, k = w.seq_lens[0], w.n_probe, w.n_layers, w.n_kv_heads, w.head_dim, w.topk
    assert (gold["seq_len"], gold["n_probe"], gold["n_layers"], gold["n_kv_heads"]) == (T, P, L, H)
    log(f"[case] full prefill routing: {L} layers, {H} KV heads, T={T}, P={P}, budget {gold['budget_bytes']}")
    tdt = torch_dtype(w.dtype)
    Kd = torch.empty((L, H, T, d), dtype=tdt, device="cuda")
    for b, h, kk, _ in gen.iter_segments(w, 0, threads=16):
        f, nb = w.blocks[b]
        Kd[f:f + nb, h].copy_(torch.from_numpy(kk).cuda().to(tdt))
    Qd = torch.empty((L, w.n_q_heads, P, d), dtype=tdt, device="cuda")
    for l in range(L):
        Qd[l].copy_(torch.from_numpy(gen.probe_queries(w, 0, layers=[l])[0]).cuda().to(tdt))
    dm = B.dims(**w.dims())
    err, _ = probe(dm, T, [Kd[l] for l in range(L)], [Qd[l] for l in range(L)], P)
    got = err.cpu().numpy()                                        # [16][8][2] fp32
    del Kd, Qd
    E2 = np.asarray(gold["E"], np.float64)                        # [128][2]
    rel = np.abs(got.reshape(-1, 2).astype(np.float64) - E2) / E2
    log(f"  losses of {len(E2)} units: worst rel error {rel.max():.2e}")
    assert rel.max() <= 2e-5
    modes, lam, st = B.route(dm, T, got, budget_bytes=gold["budget_bytes"])
    assert st == 0
    E3 = np.concatenate([E2, np.zeros((len(E2), 1))], axis=1)
    gE3 = np.concatenate([got.reshape(-1, 2).astype(np.float64), np.zeros((len(E2), 1))], axis=1)
    om = O.omega(d, k, w.dtype)
    tied = sorted({u for u, _, _ in gold["defining"]})
    log(f"  lambda* {lam:.9g} vs oracle {gold['lambda']:.9g} (unit {tied}), mix {np.bincount(modes.ravel(), minlength=3).tolist()}"
        f" vs {gold['mode_mix']}")
    assert abs(lam / gold["lambda"] - 1.0) <= 1e-4
    assert budget_defining_units(gE3, om, lam) == tied
    assert gold["near_ties"] == []
    check_modes(modes, E3, om, gold["lambda"], "prefill8b budget", exclude=tied)
    np.testing.assert_array_equal(modes.ravel(), np.asarray(gold["modes"]))


def test_fullsize_token_residual(torch_mod):
    """Token-level residual sets at the 8B shape (T = 32768, 8 KV heads, 32 query
    heads, P = 256, r = 5%): probe scores, sets, stored rows and decode of sampled
    units against the oracle, with the rules of the small token-level cases."""
    torch = torch_mod
    from paper_2607_06519_amd import binding as Bn
    from paper_2607_06519_amd.cache import CompressedCache, probe, to_device
    from test_gpu_tokres import check_token_set, score_bound, unpack_tok_unit
    from gpu_cases import TYPES, ulp_distance
    w = scaled(WORKLOADS["llama8b_tokres"], n_layers=2)
    T, G, d, H, ppm = w.seq_lens[0], w.group, w.head_dim, w.n_kv_heads, w.res_ppm
    n = O.n_residual_tokens(T, ppm)
    log(f"[case] full-size token residual: T={T} Hkv={H} Hq={w.n_q_heads} P={w.n_probe} r={ppm / 1e6} (n={n})")
    K, V = gen.layer_cache(w, 0, threads=16)
    Q = gen.probe_queries(w, 0)
    Kd, Vd, Qd = to_device(K, w.dtype), to_device(V, w.dtype), to_device(Q, w.dtype)
    dm = Bn.dims(**w.dims())
    kl, vl, ql = ([X[l] for l in range(w.n_layers)] for X in (Kd, Vd, Qd))
    _, scores = probe(dm, T, kl, ql, w.n_probe)
    got_s = scores.cpu().numpy().astype(np.float64)
    modes = np.full((1, H), O.RESIDUAL, np.uint8)
    modes[0, 0] = O.SHARED
    modes[0, H - 1] = O.EXACT
    cache = CompressedCache(dm, w.seq_lens, modes[None])
    cache.compress(0, kl, vl, token_scores=scores)
    torch.cuda.synchronize()
    del Kd, Vd, Qd
    buf = cache.host_bytes()
    q = gen.decode_queries(w, 0, scale=8.0)
    outs = [cache.decode(layer, to_device(q[layer], w.dtype)).float().cpu().numpy()[0] for layer in range(w.n_layers)]
    worst = 0.0
    for h in (0, 1, 4, H - 1):
        m = int(modes[0, h])
        got, counts = unpack_tok_unit(buf, int(cache.offsets_host[0, 0, h]), m, T, d, ppm, w.dtype, 2)
        if m == O.RESIDUAL:
            QB = Q[0:2, h * G:(h + 1) * G]
            ref_s, _ = O.token_scores(K[0:2, h], QB)
            bound = score_bound(K[0:2, h], QB)
            assert np.all(np.abs(got_s[0, h] - ref_s) <= bound), h
            S = got["TS"]
            nd = check_token_set(S, got_s[0, h], ref_s, bound, n, h)
            log(f"  head {h}: set of {n} tokens, {nd} differ from the oracle's inside the score bound")
            np.testing.assert_array_equal(counts[:-1], np.searchsorted(S, np.arange(0, T, 128)))
            assert counts[-1] == n
            ref = O.compress_unit_tokens(K[0:2, h], V[0:2, h], m, S, w.dtype)
            for key in ("MK", "MV"):
                compare_units({key: got[key]}, {key: ref[key]}, w.dtype)
            for key in ("HK", "HV"):
                assert ulp_distance(got[key], ref[key], TYPES[w.dtype][1]).max(initial=0) <= 1, key
        else:
            ref = O.compress_unit_tokens(K[0:2, h], V[0:2, h], m, None, w.dtype)
            compare_units(got, ref, w.dtype)
        for layer in range(2):
            want = O.decode_unit_tokens(ref, m, layer, q[layer][0, h * G:(h + 1) * G].astype(np.float64),
                                        1.0 / math.sqrt(d), d, 2)
            for g in range(G):
                e = rel_l2(outs[layer][h * G + g], want[g])
                worst = max(worst, e)
                assert e <= 1e-2, (h, layer, g, e)
        log(f"  unit head={h} mode={m} ok")
    log(f"  worst rel-L2 {worst:.3e}")


def test_fullsize_generation(torch_mod):
    """Generation over a 32768-token prefix at the 8B head shape: appends into a
    40-row exact tail, decode over the compressed span plus the tail (the
    several-part launch), one refresh; refreshed modes and spans checked for
    every head, decode outputs for sampled heads of every mode at every step."""
    torch = torch_mod
    from paper_2607_06519_amd import binding as Bn
    from paper_2607_06519_amd.cache import CompressedCache, Generation, to_device
    from test_gpu_generation import _new_token
    w = scaled(WORKLOADS["llama8b"], n_layers=2)
    T, H, G, d, k, L = w.seq_lens[0], w.n_kv_heads, w.group, w.head_dim, w.topk, w.n_layers
    cap, P, steps = 40, 16, 45
    heads = (0, 1, 2, 5)
    log(f"[case] full-size generation: prefix {T}, Hkv={H} Hq={w.n_q_heads}, tail {cap}, {steps} steps")
    dm = Bn.dims(**w.dims())
    modes0 = gen.fixed_modes(w)[None].copy()
    modes0[0, 0, :3] = [0, 1, 2]
    cache = CompressedCache(dm, w.seq_lens, modes0)
    K, V = gen.layer_cache(w, 0, threads=16)
    Kd, Vd = to_device(K, w.dtype), to_device(V, w.dtype)
    cache.compress(0, [Kd[l] for l in range(L)], [Vd[l] for l in range(L)])
    torch.cuda.synchronize()
    del Kd, Vd
    spans = [{h: (O.compress_unit(K[0:2, h], V[0:2, h], int(modes0[0, 0, h]), k, w.dtype), int(modes0[0, 0, h]), 2)
              for h in heads}]
    del K, V
    g = Generation(dm, cache, cap)
    rng = np.random.default_rng(11)
    tailK = [[] for _ in range(L)]
    tailV = [[] for _ in range(L)]
    recent = [[] for _ in range(L)]
    worst, refreshes = 0.0, 0
    for step in range(steps):
        if g.full:
            Qr = [np.stack(recent[l][-P:], axis=2) for l in range(L)]           # [1][Hq][P][d]
            Kt = np.array([np.stack([r[0] for r in tailK[l]], axis=1) for l in range(L)])  # [L][H][n][d]
            Vt = np.array([np.stack([r[0] for r in tailV[l]], axis=1) for l in range(L)])
            E = np.stack([O.routing_errors(Kt[:, h], np.stack(Qr)[:, 0, h * G:(h + 1) * G], k) for h in range(H)])
            lam = separated_lambdas(E, O.omega(d, k, w.dtype, 2), n=1)[0]
            modes = g.refresh([to_device(Qr[l], w.dtype) for l in range(L)], P, lam=lam)
            refreshes += 1
            om = np.stack([O.omega(d, k, w.dtype, 2) for _ in range(H)])
            ok = check_modes(modes[0, 0], E, om, lam, "full-size refresh")
            buf = g.spans[-1].host_bytes()
            span = {}
            for h in range(H):
                m = int(modes[0, 0, h])
                unit = O.compress_unit(Kt[:, h], Vt[:, h], m, k, w.dtype)
                compare_units(unpack_unit(buf, int(g.spans[-1].offsets_host[0, 0, h]), m, cap, d, k, w.dtype, 2),
                              unit, w.dtype)
                span[h] = (unit, m, 2)
            spans.append(span)
            tailK = [[] for _ in range(L)]
            tailV = [[] for _ in range(L)]
            log(f"  refresh: modes {np.bincount(modes.ravel(), minlength=3).tolist()}, {ok} checked")
        kn, vn = _new_token(w, rng)
        qs = gen.decode_queries(w, step, scale=4.0)
        for layer in range(L):
            g.append(layer, to_device(kn[layer], w.dtype), to_device(vn[layer], w.dtype))
            out = g.decode(layer, to_device(qs[layer], w.dtype)).float().cpu().numpy()
            tailK[layer].append(kn[layer])
            tailV[layer].append(vn[layer])
            for h in heads:
                tk = np.stack([r[0, h] for r in tailK[layer]])
                tv = np.stack([r[0, h] for r in tailV[layer]])
                want = O.decode_spans([sp[h] for sp in spans], tk, tv, layer,
                                      qs[layer][0, h * G:(h + 1) * G].astype(np.float64), 1.0 / math.sqrt(d), d)
                for gg in range(G):
                    e = rel_l2(out[0, h * G + gg], want[gg])
                    worst = max(worst, e)
                    assert e <= 1e-2, (step, layer, h, gg, e)
            recent[layer].append(qs[layer])
        g.advance()
    assert refreshes == 1 and len(g.spans) == 2
    log(f"  {steps} steps ok; worst rel-L2 {worst:.3e}")
