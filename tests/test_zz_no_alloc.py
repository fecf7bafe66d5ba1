"""fdkv_decode_attn_static, the decode entry point that allocates nothing (its
split-K records live in the library's static device scratch), against
fdkv_decode_attn with a caller workspace on the same cache and queries: two
calls in a row, the second on a smaller input, each bit-identical to the
workspace call (the same kernels read the same records) and within the
decode bar of the oracle; a call that needs more than the static scratch is
refused on the host."""
import math
import sys

import numpy as np
import pytest

import oracle as O
from synth import WORKLOADS, gen, scaled

from gpu_cases import oracle_decode_layer, rel_l2

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def torch_dev():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU visible")
    from paper_2607_06519_amd import binding
    binding.load()
    return torch


def _cache(torch, w, modes):
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import CompressedCache, to_device
    cache = CompressedCache(B.dims(**w.dims()), w.seq_lens, modes)
    Ks = []
    for s, T in enumerate(w.seq_lens):
        if T == 0:
            Ks.append(None)
            continue
        ws_ = scaled(w, seq_lens=(T,))
        K, V = gen.layer_cache(ws_, 0)
        Kd, Vd = to_device(K, w.dtype), to_device(V, w.dtype)
        cache.compress(s, [Kd[l] for l in range(w.n_layers)], [Vd[l] for l in range(w.n_layers)])
        Ks.append((ws_, K, V))
    torch.cuda.synchronize()
    return cache, Ks


@pytest.mark.parametrize("first,second", [("bf16", "bf16"), ("bf16", "f32")])
def test_static_decode_matches_workspace_decode(torch_dev, first, second):
    torch = torch_dev
    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import to_device
    big = scaled(WORKLOADS["llama8b"], n_layers=2, seq_lens=(9000, 4100), n_needles=4, dtype=first)
    small = scaled(WORKLOADS["llama8b"], n_layers=2, n_kv_heads=2, n_q_heads=8, seq_lens=(700, 0, 33), n_needles=2,
                   dtype=second)
    assert B.decode_workspace(B.dims(**small.dims()), small.batch, small.max_seq_len) < \
        B.decode_workspace(B.dims(**big.dims()), big.batch, big.max_seq_len) <= B.decode_static_scratch_bytes()
    for w in (big, small):
        log(f"[case] static decode: lens {w.seq_lens} Hkv={w.n_kv_heads} Hq={w.n_q_heads} {w.dtype}")
        modes = np.stack([gen.fixed_modes(w, s) for s in range(w.batch)])
        n = min(3, w.n_kv_heads)
        for s in range(w.batch):
            modes[s, 0, :n] = np.roll([0, 1, 2], s)[:n]
        cache, Ks = _cache(torch, w, modes)
        qs = gen.decode_queries(w, 3, scale=8.0)
        scale = 1.0 / math.sqrt(w.head_dim)
        tol = 1e-2 if w.dtype == "bf16" else 1e-5
        for layer in range(w.n_layers):
            q = to_device(qs[layer], w.dtype)
            ref = torch.full_like(q, 7.0)
            got = torch.full_like(q, 7.0)
            cache.decode(layer, q, ref, scale)
            B.decode_attn_static(cache.dims, cache.batch, cache.seq_lens, cache.max_seq_len, cache.modes,
                                 cache.offsets, cache.buf, layer, q, got, scale)
            torch.cuda.synchronize()
            assert torch.equal(got, ref), layer
            out = got.float().cpu().numpy()
            worst = 0.0
            for s, T in enumerate(w.seq_lens):
                if T == 0:
                    assert np.all(out[s] == 0.0)
                    continue
                ws_, K, V = Ks[s]
                units = {(b, h): O.compress_unit(K[f:f + nb, h], V[f:f + nb, h], int(modes[s, b, h]), w.topk, w.dtype)
                         for b, (f, nb) in enumerate(w.blocks) for h in range(w.n_kv_heads)}
                want = oracle_decode_layer(units, modes[s], layer, qs[layer][s].astype(np.float64), ws_)
                for hq in range(w.n_q_heads):
                    e = rel_l2(out[s, hq], want[hq])
                    worst = max(worst, e)
                    assert e <= tol, (w.seq_lens, layer, s, hq, e)
            log(f"  layer {layer}: equal to the workspace call, worst rel-L2 vs oracle {worst:.2e}")


def test_static_decode_refuses_a_call_beyond_its_scratch(torch_dev):
    torch = torch_dev
    from paper_2607_06519_amd import binding as B
    w = scaled(WORKLOADS["long70b"], n_layers=2, seq_lens=(131072,) * 4)
    dm = B.dims(**w.dims())
    need = B.decode_workspace(dm, w.batch, w.max_seq_len)
    assert need > B.decode_static_scratch_bytes()
    dummy = torch.zeros(1 << 12, dtype=torch.uint8, device="cuda")   # never read: the call stops on the host
    lens = torch.zeros(w.batch, dtype=torch.int32, device="cuda")
    with pytest.raises(B.FdkvError) as ei:
        B.decode_attn_static(dm, w.batch, lens, w.max_seq_len, dummy, dummy, dummy, 0, dummy, dummy, 0.1)
    assert ei.value.status == -3 and "static scratch" in str(ei.value)
    log(f"  refused: needs {need} bytes, scratch {B.decode_static_scratch_bytes()}")
