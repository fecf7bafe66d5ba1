"""Token-level residual sets on the GPU through the C ABI, against the oracle.

The oracle's score s_t (max over probe rows of |q . (K_t - K^S_t)|) is float64.
The kernel multiplies the probe rows by the deviations rounded to bf16 (MFMA,
exact products, fp32 sums), so its score is within
    bound_t = (2^-9 + 2^-16) max_q sum_c |q_c| |dev_c|
of the oracle's (the bf16 rounding moves each deviation by at most 2^-9 of
itself; the fp32 sum of d = 128 products adds at most d 2^-24).  Which tokens
enter the set is an integer decision on those scores: the kernel's set is
exactly the top n of its own scores (ties to the lower token), tokens whose
oracle score clears the n-th largest by more than twice the largest bound are
in, those below it by as much are out, and the number of tokens whose
membership differs from the oracle's set inside that band is reported.
Everything after the selection is checked against the oracle given the GPU's
set: the routing losses within 5e-4 relative (the bf16 deviations), stored
rows within 1 ulp (blocks of four: the fp32 butterfly's 2^-21 of the
channel's largest input plus one spacing of the storage type), decode within
relative L2 1e-2 (bf16) / 1e-5 (fp32)."""
import math
import sys

import numpy as np
import pytest

import oracle as O
from synth import WORKLOADS, gen, scaled

from gpu_cases import (BYTES, TYPES, _pad, block_of, coef_plane_bytes, compare_units, quad_value_tol, rel_l2,
                       shared_plane, sharpened_queries, ulp_distance, values)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2607_06519_amd import binding
    binding.load()
    return torch


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _tok(w, **over):
    return scaled(w, topk=0, residual=1, **over)


CASES = {
    "pairs_bf16": _tok(WORKLOADS["prefill8b"], n_layers=4, n_kv_heads=2, n_q_heads=8, seq_lens=(1500,), n_probe=48,
                       res_ppm=50000),
    "quads_bf16_ragged": _tok(WORKLOADS["prefill8b"], n_layers=4, n_kv_heads=2, n_q_heads=8, seq_lens=(1111,),
                              n_probe=32, res_ppm=80000, schedule=2),
    "mixed_e4m3_d64_g2": _tok(WORKLOADS["prefill8b"], n_layers=12, n_kv_heads=2, n_q_heads=4, head_dim=64,
                              seq_lens=(700,), n_probe=20, res_ppm=100000, schedule=1, dtype="bf16_e4m3",
                              needle_channels=8),
    "quads_f32_g1": _tok(WORKLOADS["tiny"], n_layers=4, n_kv_heads=2, n_q_heads=2, seq_lens=(600,), n_probe=24,
                         res_ppm=70000, schedule=2),
    # degenerate sets: none (r = 0), and a handful of tokens in a sequence shorter than one chunk
    "pairs_f32_empty": _tok(WORKLOADS["tiny"], n_layers=2, n_kv_heads=3, n_q_heads=6, seq_lens=(200,), n_probe=16,
                            res_ppm=0),
    "pairs_bf16_short": _tok(WORKLOADS["prefill8b"], n_layers=2, n_kv_heads=3, n_q_heads=6, seq_lens=(37,),
                             n_probe=8, res_ppm=30000, n_needles=1),
    # every token in the set (each tile of the streaming pass fully masked before any logit),
    # and a one-token sequence whose only token is in the set
    "pairs_bf16_all": _tok(WORKLOADS["prefill8b"], n_layers=2, n_kv_heads=3, n_q_heads=6, seq_lens=(300,),
                           n_probe=8, res_ppm=1000000, n_needles=1),
    "quads_e4m3_t1": _tok(WORKLOADS["prefill8b"], n_layers=4, n_kv_heads=3, n_q_heads=12, seq_lens=(1,),
                          n_probe=8, res_ppm=50000, n_needles=1, schedule=2, dtype="bf16_e4m3"),
}


def score_bound(KB, QB) -> np.ndarray:
    """Per token, the largest |kernel score - float64 score| the bf16 deviations and
    fp32 sums allow: (2^-9 + 2^-16) max over probe rows of sum_c |q_c| |dev_c|."""
    dev = np.abs(O.token_deviations(KB))                     # [B][T][d]
    QB = np.abs(np.asarray(QB, np.float64))
    out = np.zeros(dev.shape[1])
    for l in range(dev.shape[0]):
        out = np.maximum(out, (QB[l].reshape(-1, QB.shape[-1]) @ dev[l].T).max(axis=0))
    return (2.0 ** -9 + 2.0 ** -16) * out


def check_token_set(S, got_s, ref_s, bound, n, what) -> int:
    """A kernel token set against the oracle's scores: exactly n tokens, ascending, the top
    n of the kernel's own scores (ties to the lower token); tokens whose oracle score
    clears the n-th largest by more than twice the largest bound are in, those below it
    by as much out.  Returns how many tokens differ from the oracle's own set."""
    S = np.asarray(S, np.int64)
    T = len(ref_s)
    assert S.size == n, (what, S.size, n)
    assert np.all(np.diff(S) > 0), what
    np.testing.assert_array_equal(S, O.residual_tokens(got_s, n), err_msg=str(what))
    if n == 0:
        return 0
    inside = np.zeros(T, bool)
    inside[S] = True
    tau = np.sort(ref_s)[::-1][n - 1]
    band = 2.0 * bound.max()
    assert not np.any((ref_s > tau + band) & ~inside), what
    assert not np.any((ref_s < tau - band) & inside), what
    want = np.zeros(T, bool)
    want[O.residual_tokens(ref_s, n)] = True
    return int((inside != want).sum())


def unpack_tok_unit(buf, off, mode, T, d, ppm, dtype, B):
    """A token-level residual segment read back (the layout of include/fdkv.h)."""
    ti, tc = TYPES[dtype]
    e, c = BYTES[ti], BYTES[tc]
    if mode != O.RESIDUAL:
        from gpu_cases import unpack_unit
        return unpack_unit(buf, off, mode, T, d, 0, dtype, B), None
    coef = coef_plane_bytes(T, d, c)
    n = O.n_residual_tokens(T, ppm)
    mo = 2 * coef
    co = mo + _pad(-(-T // 32) * 4)
    hk = co + _pad((-(-T // 128) + 1) * 4)
    hv = hk + _pad(n * (B - 1) * d * c)

    def plane(o, rows, width, kind):
        return values(buf[off + o: off + o + rows * width * BYTES[kind]].copy(), kind).reshape(rows, width)

    words = buf[off + mo: off + mo + (-(-T // 32)) * 4].copy().view("<u4")
    bits = ((words[:, None] >> np.arange(32, dtype=np.uint32)) & 1).reshape(-1)[:T]
    counts = buf[off + co: off + co + ((-(-T // 128)) + 1) * 4].copy().view("<u4").astype(np.int64)
    u = {"MK": shared_plane(buf, off, T, d, dtype), "MV": shared_plane(buf, off + coef, T, d, dtype),
         "TS": np.nonzero(bits)[0].astype(np.int64),
         "HK": plane(hk, n, (B - 1) * d, tc).reshape(n, B - 1, d), "HV": plane(hv, n, (B - 1) * d, tc).reshape(n, B - 1, d)}
    return u, counts


@pytest.mark.parametrize("name", list(CASES))
def test_token_residual_parity(torch_dev, name):
    torch = torch_dev
    from paper_2607_06519_amd import binding as Bn
    from paper_2607_06519_amd.cache import CompressedCache, probe, to_device
    w = CASES[name]
    T, P, G, d, H = w.seq_lens[0], w.n_probe, w.group, w.head_dim, w.n_kv_heads
    ppm = w.res_ppm
    n = O.n_residual_tokens(T, ppm)
    log(f"[case] token residual {name}: T={T} blocks {w.block_sizes} d={d} G={G} r={ppm / 1e6} (n={n}) {w.dtype}")
    K, V = gen.layer_cache(w, 0)
    Q = gen.probe_queries(w, 0)
    Kd, Vd, Qd = to_device(K, w.dtype), to_device(V, w.dtype), to_device(Q, w.dtype)
    dm = Bn.dims(**w.dims())
    kl, vl, ql = ([X[l] for l in range(w.n_layers)] for X in (Kd, Vd, Qd))
    err, scores = probe(dm, T, kl, ql, P)
    got_err = err.cpu().numpy().astype(np.float64)
    got_s = scores.cpu().numpy().astype(np.float64)

    # scores against the oracle's, unit by unit, within the bf16-deviation bound
    ref_s = np.zeros((w.n_blocks, H, T))
    bound = np.zeros((w.n_blocks, H, T))
    for b, (f, B) in enumerate(w.blocks):
        for h in range(H):
            QB = Q[f:f + B, h * G:(h + 1) * G]
            ref_s[b, h], _ = O.token_scores(K[f:f + B, h], QB)
            bound[b, h] = score_bound(K[f:f + B, h], QB)
    err = np.abs(got_s - ref_s)
    log(f"  scores: max error / bound {(err / np.maximum(bound, 1e-30)).max():.3f}, "
        f"max rel error {(err / np.maximum(ref_s, 1e-30)).max():.2e}")
    assert np.all(err <= bound)

    # modes: every unit residual except a few, so the compressed sets get checked everywhere
    modes = np.full((w.n_blocks, H), O.RESIDUAL, np.uint8)
    modes[0, 0] = O.SHARED
    modes[-1, -1] = O.EXACT
    cache = CompressedCache(dm, w.seq_lens, modes[None])
    cache.compress(0, kl, vl, token_scores=scores)
    torch.cuda.synchronize()
    buf = cache.host_bytes()
    units = {}
    band_diff = 0
    for b, (f, B) in enumerate(w.blocks):
        for h in range(H):
            m = int(modes[b, h])
            got, counts = unpack_tok_unit(buf, int(cache.offsets_host[0, b, h]), m, T, d, ppm, w.dtype, B)
            if m == O.RESIDUAL:
                S = got["TS"]
                band_diff += check_token_set(S, got_s[b, h], ref_s[b, h], bound[b, h], n, (b, h))
                chunk_starts = np.arange(0, T, 128)
                np.testing.assert_array_equal(counts[:-1], np.searchsorted(S, chunk_starts))
                assert counts[-1] == n
                ref = O.compress_unit_tokens(K[f:f + B, h], V[f:f + B, h], m, S, w.dtype)
                for key in ("MK", "MV"):
                    compare_units({key: got[key]}, {key: ref[key]}, w.dtype,
                                  inputs=(K[f:f + B, h], V[f:f + B, h]) if B == 4 else None)
                for key, X in (("HK", K), ("HV", V)):
                    if B == 4:
                        mag = np.abs(X[f:f + B, h][:, S]).max(axis=0)[:, None, :]
                        assert np.all(np.abs(got[key] - ref[key]) <= quad_value_tol(ref[key], mag, TYPES[w.dtype][1]))
                    else:
                        assert ulp_distance(got[key], ref[key], TYPES[w.dtype][1]).max(initial=0) <= 1, key
                # routing losses, given the GPU's set
                E = O.routing_errors_tokens(K[f:f + B, h], Q[f:f + B, h * G:(h + 1) * G], 0)   # E_S (S empty)
                Ks = O.candidate_keys(K[f:f + B, h], O.SHARED, 0)
                Qh = Q[f:f + B, h * G:(h + 1) * G].astype(np.float64)
                contrib = sum(np.sum((Qh[l].reshape(-1, d) @ (Ks[l, S] - K[f + l, h, S]).T) ** 2) / (P * d)
                              for l in range(B)) / (B * G)
                want = np.array([E[O.SHARED], E[O.SHARED] - contrib])
                # a set of every token leaves E_R = 0: compare it on the scale of E_S
                relE = np.abs(got_err[b, h] - want) / np.maximum(np.abs(want), 1e-6 * abs(want[0]) + 1e-30)
                assert relE.max() <= 5e-4, (b, h, got_err[b, h], want)
                units[(b, h)] = ref
            else:
                units[(b, h)] = O.compress_unit_tokens(K[f:f + B, h], V[f:f + B, h], m, None, w.dtype)
    log(f"  compress ok: every set has {n} tokens ({band_diff} tokens differ from the oracle's sets, all inside "
        f"the bound), rows within 1 ulp, losses within 5e-4")

    tol = 1e-5 if w.dtype == "f32" else 1e-2
    worst = 0.0
    for qi, qs in enumerate(sharpened_queries(w, 0, K)):
        for layer in range(w.n_layers):
            out = cache.decode(layer, to_device(qs[layer], w.dtype)).float().cpu().numpy()[0]
            bi, f, B = block_of(w, layer)
            for h in range(H):
                want = O.decode_unit_tokens(units[(bi, h)], int(modes[bi, h]), layer,
                                            qs[layer][0, h * G:(h + 1) * G].astype(np.float64), 1.0 / math.sqrt(d), d, B)
                for g in range(G):
                    e = rel_l2(out[h * G + g], want[g])
                    worst = max(worst, e)
                    assert e <= tol, (name, qi, layer, h, g, e)
    log(f"  decode ok; worst rel-L2 {worst:.3e} (tol {tol})")


RATE_CASES = {
    "pairs_bf16_rates": _tok(WORKLOADS["prefill8b"], n_layers=4, n_kv_heads=4, n_q_heads=8, seq_lens=(1200,),
                             n_probe=32, res_ppm=0, res_rates=(20000, 50000, 150000)),
    "mixed_bf16_rates": _tok(WORKLOADS["prefill8b"], n_layers=12, n_kv_heads=2, n_q_heads=4, head_dim=64,
                             seq_lens=(700,), n_probe=20, res_ppm=0, res_rates=(10000, 40000, 100000, 300000),
                             schedule=1, needle_channels=8),
}
# byte budgets, as a fraction of the way from all-shared to all-exact, at which the seeded
# cases route with every other unit at least 2e-3 from a tie (checked in the test)
RATE_BUDGET = {"pairs_bf16_rates": 0.35, "mixed_bf16_rates": 0.4}


@pytest.mark.parametrize("name", list(RATE_CASES))
def test_token_rates_routed_per_unit(torch_dev, name):
    """Token-level sets whose fraction is routed per residual head (Section 3: r_{b,h} by the
    routing loss budget): the probe's E_S and E_R at every candidate fraction against the
    oracle (given the kernel's sets: the top n_j of its own scores), the budget routing over
    (mode, fraction) against the oracle's on its own float64 losses (units within 1e-3 of a
    tie would be near-ties at the bf16-deviation precision of these losses, and must be
    absent), then compress and decode with each unit's own fraction."""
    torch = torch_dev
    from paper_2607_06519_amd import binding as Bn
    from paper_2607_06519_amd.cache import CompressedCache, probe, to_device
    from gpu_cases import check_modes
    w = RATE_CASES[name]
    T, P, G, d, H = w.seq_lens[0], w.n_probe, w.group, w.head_dim, w.n_kv_heads
    rates = list(w.res_rates)
    J = len(rates)
    log(f"[case] routed fractions {name}: T={T} blocks {w.block_sizes} rates {rates}")
    K, V = gen.layer_cache(w, 0)
    Q = gen.probe_queries(w, 0)
    Kd, Vd, Qd = to_device(K, w.dtype), to_device(V, w.dtype), to_device(Q, w.dtype)
    dm = Bn.dims(**w.dims())
    kl, vl, ql = ([X[l] for l in range(w.n_layers)] for X in (Kd, Vd, Qd))
    err, scores = probe(dm, T, kl, ql, P)
    got_err = err.cpu().numpy().astype(np.float64)                 # [nb][H][1 + J]
    got_s = scores.cpu().numpy().astype(np.float64)
    assert got_err.shape == (w.n_blocks, H, 1 + J)
    E_or = np.zeros((w.n_blocks, H, 1 + J))
    worst = 0.0
    for b, (f, B) in enumerate(w.blocks):
        for h in range(H):
            QB = Q[f:f + B, h * G:(h + 1) * G]
            E_or[b, h] = O.routing_errors_token_rates(K[f:f + B, h], QB, rates)
            Ks = O.candidate_keys(K[f:f + B, h], O.SHARED, 0)
            want = [E_or[b, h, 0]]
            for r in rates:
                S = O.residual_tokens(got_s[b, h], O.n_residual_tokens(T, r))
                contrib = sum(np.sum((QB[l].astype(np.float64).reshape(-1, d) @ (Ks[l, S] - K[f + l, h, S]).T) ** 2)
                              / (P * d) for l in range(B)) / (B * G)
                want.append(E_or[b, h, 0] - contrib)
            want = np.array(want)
            rel = np.abs(got_err[b, h] - want) / np.maximum(np.abs(want), 1e-6 * want[0])
            worst = max(worst, rel.max())
            assert rel.max() <= 5e-4, (b, h, got_err[b, h], want)
    log(f"  losses at {J} fractions within {worst:.2e} of the oracle given the kernel's sets")
    # the byte budget: a set fraction of the way from all-shared to all-exact
    sizes = [B for B in w.block_sizes for _ in range(H)]
    lo = sum(O.unit_bytes_tokens(O.SHARED, T, d, 0, w.dtype, B) for B in sizes)
    hi = sum(O.unit_bytes_tokens(O.EXACT, T, d, 0, w.dtype, B) for B in sizes)
    budget = int(lo + RATE_BUDGET[name] * (hi - lo))
    modes, lam, st = Bn.route(dm, T, got_err.astype(np.float32), budget_bytes=budget)
    assert st == 0
    om_modes, om_r, om_lam, ok = O.route_token_rates(E_or.reshape(-1, 1 + J), T, d, rates, w.dtype,
                                                      budget=budget, unit_sizes=sizes)
    assert ok
    cand = [O.token_rate_candidates(d, rates, w.dtype, B) for B in sizes]
    om = np.stack([c[0] for c in cand])
    Ec = np.concatenate([E_or.reshape(-1, 1 + J), np.zeros((len(sizes), 1))], axis=1)
    # compare the choices as candidate indices (shared 0, residual at r_j 1 + j, exact J + 1)
    def to_cand(byte):
        m = int(byte) & 3
        return 0 if m == 0 else J + 1 if m == 2 else 1 + (int(byte) >> 2)
    got_c = np.array([to_cand(x) for x in modes.ravel()])
    from gpu_cases import budget_defining_units
    tied = budget_defining_units(Ec, om, om_lam)
    gEc = np.concatenate([got_err.reshape(-1, 1 + J).astype(np.float32).astype(np.float64),
                          np.zeros((len(sizes), 1))], axis=1)
    assert budget_defining_units(gEc, om, lam) == tied, (tied, budget_defining_units(gEc, om, lam))
    assert abs(lam / om_lam - 1.0) <= 2e-3, (lam, om_lam)
    check_modes(got_c, Ec, om, om_lam, f"{name} (mode, fraction)", exclude=tied, near=1e-3)
    want_c = O.route(Ec, om, om_lam)
    np.testing.assert_array_equal(got_c[tied], want_c[tied])
    log(f"  routed: lambda {lam:.5g} (oracle {om_lam:.5g}), modes {np.bincount(modes.ravel() & 3, minlength=3).tolist()}, "
        f"fractions of residual heads {np.bincount(modes.ravel()[(modes.ravel() & 3) == 1] >> 2, minlength=J).tolist()}")
    # compress and decode with each unit's own fraction
    cache = CompressedCache(dm, w.seq_lens, modes[None])
    cache.compress(0, kl, vl, token_scores=scores)
    torch.cuda.synchronize()
    buf = cache.host_bytes()
    units = {}
    for b, (f, B) in enumerate(w.blocks):
        for h in range(H):
            byte = int(modes[b, h])
            m = byte & 3
            ppm = rates[byte >> 2] if m == 1 else 0
            n = O.n_residual_tokens(T, ppm)
            got, counts = unpack_tok_unit(buf, int(cache.offsets_host[0, b, h]), m, T, d, ppm, w.dtype, B)
            if m == O.RESIDUAL:
                S = got["TS"]
                QB = Q[f:f + B, h * G:(h + 1) * G]
                check_token_set(S, got_s[b, h], O.token_scores(K[f:f + B, h], QB)[0], score_bound(K[f:f + B, h], QB),
                                n, (b, h))
                np.testing.assert_array_equal(counts[:-1], np.searchsorted(S, np.arange(0, T, 128)))
                assert counts[-1] == n
                units[(b, h)] = O.compress_unit_tokens(K[f:f + B, h], V[f:f + B, h], m, S, w.dtype)
            else:
                units[(b, h)] = O.compress_unit_tokens(K[f:f + B, h], V[f:f + B, h], m, None, w.dtype)
    worst = 0.0
    for qs in sharpened_queries(w, 0, K):
        for layer in range(w.n_layers):
            out = cache.decode(layer, to_device(qs[layer], w.dtype)).float().cpu().numpy()[0]
            bi, f, B = block_of(w, layer)
            for h in range(H):
                want = O.decode_unit_tokens(units[(bi, h)], int(modes[bi, h]) & 3, layer,
                                            qs[layer][0, h * G:(h + 1) * G].astype(np.float64), 1.0 / math.sqrt(d), d, B)
                for g in range(G):
                    e = rel_l2(out[h * G + g], want[g])
                    worst = max(worst, e)
                    assert e <= 1e-2, (name, layer, h, g, e)
    log(f"  compress and decode with per-unit fractions ok; worst rel-L2 {worst:.3e}")


GEN_CASES = {
    "pairs_bf16_gen": _tok(WORKLOADS["prefill8b"], n_layers=4, n_kv_heads=2, n_q_heads=8, seq_lens=(600,),
                           n_probe=16, res_ppm=100000),
    # one block of four: three heads, so the prefix holds a shared, a token-set and an exact unit
    "quads_e4m3_gen": _tok(WORKLOADS["prefill8b"], n_layers=4, n_kv_heads=3, n_q_heads=12, seq_lens=(400,),
                           n_probe=16, res_ppm=100000, schedule=2, dtype="bf16_e4m3"),
}


@pytest.mark.parametrize("name", list(GEN_CASES))
def test_token_sets_in_generation(torch_dev, name):
    """Decode over spans that hold token-level sets (the prefix, then two refreshed tails) and
    the exact tail, i.e. the multi-part decode of a generation: against attention over the
    oracle's reconstruction of every span (Eq. 3 with the GPU's own sets, whose validity
    test_token_residual_parity checks) followed by the tail rows."""
    torch = torch_dev
    from paper_2607_06519_amd import binding as Bn
    from paper_2607_06519_amd.cache import CompressedCache, Generation, probe, to_device
    from test_gpu_generation import _new_token
    w = GEN_CASES[name]
    T, P, G, d, H, L = w.seq_lens[0], w.n_probe, w.group, w.head_dim, w.n_kv_heads, w.n_layers
    ppm, cap, steps = w.res_ppm, 24, 2 * 24 + 3
    log(f"[case] token sets in generation {name}: prefix {T}, tail {cap}, {steps} steps, blocks {w.block_sizes} "
        f"{w.dtype}")
    dm = Bn.dims(**w.dims())
    K, V = gen.layer_cache(w, 0)
    Q = gen.probe_queries(w, 0)
    Kd, Vd, Qd = to_device(K, w.dtype), to_device(V, w.dtype), to_device(Q, w.dtype)
    kl, vl, ql = ([X[l] for l in range(L)] for X in (Kd, Vd, Qd))
    _, scores = probe(dm, T, kl, ql, P)
    modes = np.full((w.n_blocks, H), O.RESIDUAL, np.uint8)
    modes[0, 0] = O.SHARED
    modes[-1, -1] = O.EXACT
    cache = CompressedCache(dm, w.seq_lens, modes[None])
    cache.compress(0, kl, vl, token_scores=scores)
    torch.cuda.synchronize()

    def span_units(span, smodes, KX, VX, n_tok):
        """(unit, mode, B) per (block, head): the oracle's unit built on the span's own set."""
        buf = span.host_bytes()
        units = {}
        for b, (f, B) in enumerate(w.blocks):
            for h in range(H):
                m = int(smodes[b, h])
                got, _ = unpack_tok_unit(buf, int(span.offsets_host[0, b, h]), m, n_tok, d, ppm, w.dtype, B)
                S = got["TS"] if m == O.RESIDUAL else None
                if m == O.RESIDUAL:
                    assert S.size == O.n_residual_tokens(n_tok, ppm), (b, h, S.size)
                units[(b, h)] = (O.compress_unit_tokens(KX[f:f + B, h], VX[f:f + B, h], m, S, w.dtype), m, B)
        return units

    spans = [span_units(cache, modes, K, V, T)]
    g = Generation(dm, cache, cap)
    rng = np.random.default_rng(11)
    tailK, tailV, recent = ([[] for _ in range(L)] for _ in range(3))
    blk = {l: (b, f, B) for b, (f, B) in enumerate(w.blocks) for l in range(f, f + B)}
    tol = 1e-2
    worst, refreshes, n_res = 0.0, 0, int((modes == O.RESIDUAL).sum())
    for step in range(steps):
        if g.full:
            probe_rows = [to_device(np.stack(recent[l][-P:], axis=2), w.dtype) for l in range(L)]
            # a byte budget halfway between the all-shared and the all-exact tail span routes a mix
            size = lambda m: sum(O.unit_bytes_tokens(m, cap, d, ppm, w.dtype, B) for _, B in w.blocks) * H
            budget = (size(O.SHARED) + size(O.EXACT)) // 2
            new_modes = g.refresh(probe_rows, P, budget_bytes=budget)[0]
            refreshes += 1
            n_res += int(((new_modes & 3) == O.RESIDUAL).sum())
            Kt = np.stack([np.stack(tailK[l], axis=2)[0] for l in range(L)])   # [L][H][cap][d]
            Vt = np.stack([np.stack(tailV[l], axis=2)[0] for l in range(L)])
            spans.append(span_units(g.spans[-1], new_modes & 3, Kt, Vt, cap))
            tailK, tailV = [[] for _ in range(L)], [[] for _ in range(L)]
            log(f"  refresh {refreshes}: modes {np.bincount((new_modes & 3).ravel(), minlength=3).tolist()}")
        kn, vn = _new_token(w, rng)
        qs = gen.decode_queries(w, step, scale=4.0)
        for layer in range(L):
            g.append(layer, to_device(kn[layer], w.dtype), to_device(vn[layer], w.dtype))
            out = g.decode(layer, to_device(qs[layer], w.dtype)).float().cpu().numpy()[0]
            tailK[layer].append(kn[layer])
            tailV[layer].append(vn[layer])
            b, f, B = blk[layer]
            for h in range(H):
                Ks, Vs = [], []
                for span in spans:
                    unit, m, _ = span[(b, h)]
                    Ks.append(O.reconstruct_layer_tokens(unit, m, layer - f, d, "K", B))
                    Vs.append(O.reconstruct_layer_tokens(unit, m, layer - f, d, "V", B))
                Ks.append(np.stack([r[0, h] for r in tailK[layer]]).astype(np.float64))
                Vs.append(np.stack([r[0, h] for r in tailV[layer]]).astype(np.float64))
                want = O.attention(qs[layer][0, h * G:(h + 1) * G].astype(np.float64), np.concatenate(Ks),
                                   np.concatenate(Vs), 1.0 / math.sqrt(d))
                for gg in range(G):
                    e = rel_l2(out[h * G + gg], want[gg])
                    worst = max(worst, e)
                    assert e <= tol, (name, step, layer, h, gg, e)
            recent[layer].append(qs[layer])
        g.advance()
    assert refreshes == 2 and len(g.spans) == 3
    log(f"  {steps} steps ok; worst rel-L2 {worst:.3e} (tol {tol}); {n_res} token-set units over the spans")
