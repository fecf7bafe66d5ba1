"""Writes prefill8b_routing.json: the oracle's routing of the 8B prefill
workload (32 layers in pairs, 8 KV heads, 32 query heads, T = 32768, 256
probe rows per query head, bf16, top-16).

For every (pair, KV head) unit it stores Eq. (2)'s losses E_S and E_R from
``oracle.routing_errors`` (the literal two-logit-matrix form, fp64), then the
budget rule of Section 3 (``oracle.route_budget``) with the byte budget of the
workload's seeded 50/35/15 shared/residual/exact mix: the modes, lambda*, the
unit and mode pair whose breakpoint lambda* is, and the smallest relative cost
margin of every other unit at lambda* (near-ties are margins below 1e-4).

Only the oracle and the seeded generator are called:
    python tests/golden/make_prefill8b_routing.py [--threads N]
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time
from concurrent.futures import ThreadPoolExecutor

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import oracle as O  # noqa: E402
from synth import WORKLOADS, gen  # noqa: E402

OUT = os.path.join(os.path.dirname(os.path.abspath(__file__)), "prefill8b_routing.json")


def unit_errors(w, b, h):
    K, _, _ = gen.block_segment(w, 0, b, h)
    f, B = w.blocks[b]
    G = w.group
    Q = gen.probe_queries(w, 0, layers=list(range(f, f + B)))[:, h * G:(h + 1) * G]
    return O.routing_errors(K, Q, w.topk)


def margins_at(E, om, lam):
    """Relative cost margin of every unit's chosen mode at lam: min over the other
    modes of (cost' - cost) / cost (inf when the chosen cost is 0)."""
    cost = E + lam * om
    modes = O.route(E, om, lam)
    out = np.empty(len(E))
    for u, m in enumerate(modes):
        others = [cost[u, j] for j in range(3) if j != m]
        c = cost[u, m]
        out[u] = min(others) / c - 1.0 if c > 0 else math.inf
    return modes, out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--threads", type=int, default=4)
    args = ap.parse_args()
    w = WORKLOADS["prefill8b"]
    T, d, k = w.seq_lens[0], w.head_dim, w.topk
    units = [(b, h) for b in range(w.n_blocks) for h in range(w.n_kv_heads)]
    t0 = time.time()
    with ThreadPoolExecutor(max_workers=args.threads) as ex:
        E = np.array(list(ex.map(lambda u: unit_errors(w, *u), units)))
    print(f"losses of {len(units)} units in {time.time() - t0:.0f}s", flush=True)
    budget = O.cache_bytes([T], gen.fixed_modes(w, 0)[None], d, k, w.dtype)
    modes, lam, ok = O.route_budget(E, T, d, k, w.dtype, budget)
    assert ok
    om = O.omega(d, k, w.dtype)
    # the unit and mode pair whose breakpoint lambda* is
    defining = []
    for u in range(len(E)):
        for a, b in ((0, 1), (1, 2), (0, 2)):
            if (E[u, a] - E[u, b]) / (om[b] - om[a]) == lam:
                defining.append([u, a, b])
    _, marg = margins_at(E, om, lam)
    others = [u for u in range(len(E)) if u not in {x[0] for x in defining}]
    near = [u for u in others if marg[u] < 1e-4]
    rec = {
        "workload": w.name, "seq_len": T, "n_probe": w.n_probe, "head_dim": d, "topk": k, "dtype": w.dtype,
        "n_layers": w.n_layers, "n_kv_heads": w.n_kv_heads, "n_q_heads": w.n_q_heads,
        "budget_bytes": int(budget), "lambda": lam,
        "E": E[:, :2].tolist(), "modes": [int(m) for m in modes], "mode_mix": np.bincount(modes, minlength=3).tolist(),
        "defining": defining, "min_margin_others": float(min(marg[u] for u in others)),
        "near_ties": near,
        "source": "oracle.routing_errors (literal Eq. 2, fp64) and oracle.route_budget",
    }
    with open(OUT, "w") as f:
        json.dump(rec, f, indent=1)
    print(f"lambda* {lam:.6g} by {defining}, mix {rec['mode_mix']}, near-ties {near}, "
          f"min margin of the others {rec['min_margin_others']:.3g}", flush=True)


if __name__ == "__main__":
    main()
