#!/usr/bin/env python3
"""Benchmark of the compressed-KV decode path on one MI355X.

A step is one decode token through every layer of the workload (default:
the Llama-3-8B-shaped cache, 32 layers, 32 query heads on 8 KV heads,
d = 128, 32768 cached tokens, bf16, top-16 residuals, seeded 64/45/19
shared/residual/exact head mix).  Inputs are resident in HBM before timing.
Layers run in cold order (all even layers, then all odd ones) so the shared
planes of a pair are evicted from the 256 MB Infinity Cache before the pair's
second layer re-reads them; the headline bandwidth is therefore HBM
bandwidth.  The step is captured once in a HIP graph and replayed: by default
10 untimed steps, then 100 timed together (the mean is `value`), then the same
100 again each between its own events (p50 and p95 in `step_ms_stats`).

Printed: one JSON line with the metric, a roofline object for the decode
launch (split-K + combine per layer, timed with HIP events on the launch
stream), the prefill path (probe, route, compress) timed on the same cache,
the CPU oracle timed on a bounded sample of the same workload, and (for the
default workload) the decode lines of the 16-sequence batch and the 70B-shaped
131k-token cache, each measured by a child process before this one starts
(`other_workloads`).
"""
from __future__ import annotations

import argparse
import hashlib
import re
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama8b")
    ap.add_argument("--order", choices=["cold", "model"], default="cold")
    ap.add_argument("--no-graph", action="store_true")
    ap.add_argument("--no-prefill", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--threads", type=int, default=16)
    ap.add_argument("--gen-tail", type=int, default=512,
                    help="generation leg: exact-tail rows between refreshes (0 skips the leg)")
    ap.add_argument("--calibrate-copy-mib", type=int, default=0,
                    help="before timing, copy this many MiB device-to-device once (a copy kernel of known "
                         "size that calibrates rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    ap.add_argument("--summarize-trace", metavar="CSV",
                    help="print a per-kernel summary of a rocprofv3 kernel-trace CSV and exit")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print HBM bytes per dispatch from rocprofv3 FETCH_SIZE and WRITE_SIZE counter CSVs, "
                         "scaled by the calibration copy, and exit")
    ap.add_argument("--traffic-json", metavar="PATH", help="with --summarize-pmc: also write the decode "
                    "traffic record that the bench line reads")
    ap.add_argument("--legs", default=None,
                    help="comma-separated further decode workloads measured in child processes before this "
                         "one and reported under other_workloads (default: batched8b,long70b for the llama8b "
                         "run, none otherwise; 'none' skips them)")
    return ap.parse_args()


def run_legs(names, args):
    """Decode-only bench lines of further workloads, each a child process of this script started
    before this process touches the GPU; returns a compact record per workload."""
    import subprocess
    out = {}
    for wl in names:
        cmd = [sys.executable, os.path.abspath(__file__), "--workload", wl, "--no-prefill", "--no-cpu-baseline",
               "--gen-tail", "0", "--steps", str(min(args.steps, 20)), "--warmup", str(min(args.warmup, 3)),
               "--legs", "none"]
        log(f"[bench] leg {wl}: {' '.join(cmd[1:])}")
        r = subprocess.run(cmd, stdout=subprocess.PIPE, text=True, timeout=600)
        if r.returncode != 0:
            raise RuntimeError(f"bench leg {wl} failed with status {r.returncode}")
        d = json.loads(r.stdout.strip().splitlines()[-1])
        rf = d["roofline"]
        out[wl] = {"value": d["value"], "unit": d["unit"], "ms_per_step": d["ms_per_step"],
                   "steps": d["steps"], "dtype": d["dtype"],
                   "launch_us": rf["launch_us"], "frac": rf["frac"], "achieved_gbs": rf["achieved"],
                   "bytes_per_launch": rf["bytes_per_launch"], "traffic": rf["traffic"],
                   "config": {k: d["config"][k] for k in ("n_layers", "n_kv_heads", "n_q_heads", "head_dim",
                                                          "batch", "seq_len", "mode_mix", "cache_gb")}}
    return out


def bytes_per_token(mode, d, k, e, c, B=2):
    """Algorithmic bytes one decode layer reads per token of a head: the two
    dense planes (shared coefficients of c bytes, or exact K/V of e bytes)
    plus, for residual heads, k (index, value) pairs for K and for V (1-byte
    channels in pairs, 2-byte codes in blocks of four)."""
    if mode == 2:
        return 2 * d * e
    return 2 * d * c if mode == 0 else 2 * d * c + 2 * k * ((1 if B == 2 else 2) + c)


def unit_ppm(w, byte):
    """The token-level set's fraction (ppm) of a unit with mode byte ``byte``."""
    return w.res_rates[(int(byte) >> 2) & 7] if w.res_rates else w.res_ppm


def unit_read_bytes(w, mode, T, B):
    """Algorithmic bytes one decode layer reads from one (block, KV head) unit of T
    tokens.  With token-level residual sets a residual unit is read as its two
    shared planes, the token mask (one bit per token), the running counts (one
    word per 128 tokens, plus the total) and every high-frequency row of its n
    tokens (B - 1 rows of K and of V each)."""
    d, e, c = w.head_dim, w.elem_bytes, w.coef_bytes
    ppm = unit_ppm(w, mode)
    mode &= 3                                    # bits 2-4 of a mode byte: the routed fraction
    if w.residual != 1 or mode != 1:
        return T * bytes_per_token(mode, d, w.topk, e, c, B)
    n = (T * ppm + 999999) // 1000000
    return T * 2 * d * c + -(-T // 32) * 4 + (-(-T // 128) + 1) * 4 + n * 2 * (B - 1) * d * c


def code_tokens(text):
    """C++ source without comments and whitespace: edits to comments keep the hash."""
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    return " ".join(text.split())


def kernel_source_hash(read=None):
    """Hash of the code the decode kernels build from; counter runs recorded under another hash
    are not used.  ``read(name)`` returns a file's text (default: the working tree)."""
    if read is None:
        def read(name):
            with open(os.path.join(ROOT, "paper_2607_06519_amd", "csrc", name)) as f:
                return f.read()
    h = hashlib.sha256()
    for name in ("decode.hip", "decode_stream.hip", "fdkv_common.h", "fdkv_kernels.h"):
        h.update(code_tokens(read(name)).encode())
    return h.hexdigest()[:16]


def load_traffic(workload):
    """HBM bytes per launch from committed rocprofv3 counter runs, if they match this kernel source."""
    path = os.path.join(ROOT, "profiles", f"decode_{workload}_traffic.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("source_hash") != kernel_source_hash():
        return None
    return t.get("bytes_per_launch")


def summarize_trace(path):
    """Per-kernel count / mean / total duration from a rocprofv3 kernel-trace CSV."""
    import csv
    from collections import defaultdict
    dur = defaultdict(list)
    with open(path) as f:
        for r in csv.DictReader(f):
            dur[r["Kernel_Name"]].append((int(r["End_Timestamp"]) - int(r["Start_Timestamp"])) * 1e-3)
    rows = sorted(dur.items(), key=lambda kv: -sum(kv[1]))
    print(f"{'calls':>7} {'mean_us':>10} {'min_us':>9} {'max_us':>9} {'total_ms':>10}  kernel")
    for name, v in rows:
        print(f"{len(v):7d} {sum(v) / len(v):10.2f} {min(v):9.2f} {max(v):9.2f} {sum(v) * 1e-3:10.3f}  {name[:110]}")


def summarize_pmc(fetch_csv, write_csv, traffic_json=None, workload="llama8b"):
    """Mean FETCH_SIZE / WRITE_SIZE per dispatch and kernel, scaled by the calibration copy."""
    import csv
    from collections import defaultdict

    def read(path, counter):
        out = defaultdict(list)
        with open(path) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] == counter:
                    out[r["Kernel_Name"]].append((float(r["Counter_Value"]) * 1024.0, int(r["Grid_Size"])))
        return out

    fetch, write = read(fetch_csv, "FETCH_SIZE"), read(write_csv, "WRITE_SIZE")
    # the calibration copy: the largest torch copy kernel dispatch (reads and writes N bytes each)
    cal_name = max((k for k in fetch if "copy" in k.lower() or "elementwise" in k.lower()),
                   key=lambda k: max(v for v, _ in fetch[k]), default=None)
    cal_f = max(v for v, _ in fetch[cal_name]) if cal_name else None
    cal_w = max(v for v, _ in write.get(cal_name, [(0.0, 0)])) if cal_name else None
    print(f"calibration kernel: {cal_name[:80] if cal_name else None}")
    print(f"  FETCH_SIZE {cal_f:.4g} B, WRITE_SIZE {cal_w:.4g} B per dispatch")
    print(f"{'calls':>6} {'fetch_MB':>10} {'write_MB':>10}  kernel  (raw counter bytes per dispatch)")
    for name in sorted(fetch, key=lambda k: -sum(v for v, _ in fetch[k])):
        fv = [v for v, _ in fetch[name]]
        wv = [v for v, _ in write.get(name, [])] or [0.0]
        print(f"{len(fv):6d} {sum(fv) / len(fv) / 1e6:10.3f} {sum(wv) / len(wv) / 1e6:10.3f}  {name[:100]}")
    return cal_name, cal_f, cal_w, fetch, write


def main():
    args = parse()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_pmc:
        cal_name, cal_f, cal_w, fetch, write = summarize_pmc(*args.summarize_pmc)
        if args.traffic_json and args.calibrate_copy_mib > 0 and cal_f:
            n = args.calibrate_copy_mib << 20
            fs, ws_ = n / cal_f, n / cal_w
            def per_dispatch(names):
                fb = sum(sum(v for v, _ in fetch[k]) / len(fetch[k]) for k in names) * fs
                wb = sum(sum(v for v, _ in write[k]) / len(write[k]) for k in names if k in write) * ws_
                return fb, wb
            dec = [k for k in fetch if "decode_stream" in k or "decode_splitk" in k]   # the split-K launch
            mrg = [k for k in fetch if "decode_merge" in k]
            fb, wb = per_dispatch(dec)
            mf, mw = per_dispatch(mrg)
            rec = {"source_hash": kernel_source_hash(), "bytes_per_launch": fb + wb, "fetch_bytes": fb,
                   "write_bytes": wb, "kernels": dec, "combine_bytes": mf + mw, "fetch_scale": fs,
                   "write_scale": ws_, "calibration_bytes": n}
            with open(args.traffic_json, "w") as f:
                json.dump(rec, f, indent=1)
            print(f"split-K launch traffic: fetch {fb / 1e6:.2f} MB + write {wb / 1e6:.2f} MB per layer; combine "
                  f"{(mf + mw) / 1e6:.3f} MB (scales {fs:.4f}, {ws_:.4f})")
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the compressed-KV path here has no multi-GPU leg "
              f"(asked for --gpus {args.gpus}); run with --gpus 1", file=sys.stderr)
        sys.exit(2)
    legs = args.legs
    if legs is None:
        legs = "batched8b,long70b" if args.workload == "llama8b" else "none"
    other = run_legs([x for x in legs.split(",") if x and x != "none"], args) if legs != "none" else None

    import numpy as np
    import torch

    from paper_2607_06519_amd import binding as B
    from paper_2607_06519_amd.cache import CompressedCache, probe, torch_dtype
    from synth import WORKLOADS, gen

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    B.load()
    w = WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    L, H, Hq, d, k = w.n_layers, w.n_kv_heads, w.n_q_heads, w.head_dim, w.topk
    e = w.elem_bytes
    tdt = torch_dtype(w.dtype)
    dm = B.dims(**w.dims())

    # ------------------------------------------------------------ inputs in HBM
    t0 = time.time()
    Ks, Vs = [], []
    for s in range(w.batch):
        T = w.seq_lens[s]
        Kd = torch.empty((L, H, T, d), dtype=tdt, device=dev)
        Vd = torch.empty((L, H, T, d), dtype=tdt, device=dev)
        for b, h, kk, vv in gen.iter_segments(w, s, threads=args.threads):
            f, nb = w.blocks[b]
            Kd[f:f + nb, h].copy_(torch.from_numpy(kk).to(dev).to(tdt))
            Vd[f:f + nb, h].copy_(torch.from_numpy(vv).to(dev).to(tdt))
        Ks.append(Kd)
        Vs.append(Vd)
    torch.cuda.synchronize()
    log(f"[bench] generated {w.name} K/V in {time.time() - t0:.1f}s")

    if args.calibrate_copy_mib > 0:
        n = args.calibrate_copy_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device=dev)
        dst = torch.empty(n, dtype=torch.uint8, device=dev)
        src.fill_(1)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {n} bytes")
        del src, dst

    modes = np.stack([gen.fixed_modes(w, s) for s in range(w.batch)])
    all_scores = []
    if w.residual == 1:                         # token-level sets need the probe's token scores
        for s in range(w.batch):
            qp = [torch.from_numpy(gen.probe_queries(w, s, layers=[l])[0]).to(dev).to(tdt) for l in range(L)]
            errs, scores = probe(dm, w.seq_lens[s], [Ks[s][l] for l in range(L)], qp, w.n_probe)
            if w.res_rates:
                # fractions routed per residual head: the probe's losses under the budget of the seeded mix
                # with every residual head at the middle candidate fraction
                mid = np.where(modes[s] == 1, 1 | ((len(w.res_rates) // 2) << 2), modes[s]).astype(np.uint8)
                _, budget = B.layout(dm, [w.seq_lens[s]], mid[None])
                modes[s], _, _ = B.route(dm, w.seq_lens[s], errs.cpu().numpy(), budget_bytes=budget,
                                         allow_infeasible=True)
            all_scores.append(scores)
            del qp
    cache = CompressedCache(dm, w.seq_lens, modes)
    for s in range(w.batch):
        scores = all_scores[s] if all_scores else None
        cache.compress(s, [Ks[s][l] for l in range(L)], [Vs[s][l] for l in range(L)], token_scores=scores)
    del all_scores
    torch.cuda.synchronize()
    log(f"[bench] compressed cache: {cache.total_bytes / 1e9:.3f} GB, mix {np.bincount(modes.ravel() & 3, minlength=3).tolist()}")

    # algorithmic bytes per layer launch: sum over (seq, KV head) of T * bytes per token of the head's mode
    block_of = {l: (b, l - f, nb) for b, (f, nb) in enumerate(w.blocks) for l in range(f, f + nb)}
    bytes_layer = []
    for layer in range(L):
        b, _, nb = block_of[layer]
        bytes_layer.append(sum(unit_read_bytes(w, int(modes[s, b, h]), w.seq_lens[s], nb)
                               for s in range(w.batch) for h in range(H)))
    bytes_step = sum(bytes_layer)

    # cold order: every block's first layers, then its second layers, ...: the layers that share a
    # block's planes run a whole sweep apart, so each re-read comes from HBM
    order = sorted(range(L), key=lambda l: (block_of[l][1], l)) if args.order == "cold" else list(range(L))
    n_q = args.steps + args.warmup
    qs = torch.empty((n_q, L, w.batch, Hq, d), dtype=tdt, device=dev)
    for i in range(n_q):
        qs[i].copy_(torch.from_numpy(gen.decode_queries(w, i % w.steps)).to(dev).to(tdt))
    q_static = torch.empty((L, w.batch, Hq, d), dtype=tdt, device=dev)
    out_static = torch.empty((L, w.batch, Hq, d), dtype=tdt, device=dev)
    scale = 1.0 / math.sqrt(d)

    def step(q, out):
        for layer in order:
            cache.decode(layer, q[layer], out[layer], scale)

    # ------------------------------------------------------------ decode steps
    stream = torch.cuda.Stream()
    stream.wait_stream(torch.cuda.current_stream())
    graph = None
    with torch.cuda.stream(stream):
        q_static.copy_(qs[0])
        step(q_static, out_static)
        if not args.no_graph:
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph, stream=stream):
                step(q_static, out_static)
        torch.cuda.synchronize()

        def run(i):
            q_static.copy_(qs[i])
            if graph is not None:
                graph.replay()
            else:
                step(q_static, out_static)

        for i in range(args.warmup):
            run(i)
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record(stream)
        for i in range(args.steps):
            run(args.warmup + i)
        ev1.record(stream)
        torch.cuda.synchronize()
        step_ms = ev0.elapsed_time(ev1) / args.steps
        # the per-step spread, after the timed region: the same steps again, each bracketed by its
        # own events (the mean of these includes the events themselves; `value` does not)
        sev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
        for i in range(args.steps):
            sev[i][0].record(stream)
            run(args.warmup + i)
            sev[i][1].record(stream)
        torch.cuda.synchronize()
        per_step = np.array([a.elapsed_time(b) for a, b in sev])
        step_stats = {"n": args.steps, "mean": float(per_step.mean()), "p50": float(np.percentile(per_step, 50)),
                      "p95": float(np.percentile(per_step, 95)), "min": float(per_step.min()),
                      "max": float(per_step.max())}

        # per-launch timing with HIP events on the launch stream, each phase replayed as a graph of
        # the step's L launches in cold layer order (every layer's split-K records come from HBM, as
        # in the step): the split-K launch alone (fdkv_decode_partial: decode_stream_kernel, the
        # dominant kernel), the combine launch alone (fdkv_decode_combine: decode_merge_kernel);
        # per launch = the replays' time / (replays x L).  The one-call layer decode is timed eagerly
        # with events around each call.
        n_chunks = -(-cache.max_seq_len // 512)

        def split_phase():
            for layer in order:
                B.decode_partial(dm, w.batch, cache.seq_lens, cache.max_seq_len, cache.modes, cache.offsets,
                                 cache.buf, layer, q_static[layer], scale, cache.ws, stream)

        def combine_phase():
            for layer in order:
                B.decode_combine(dm, w.batch, n_chunks, out_static[layer], cache.ws, stream)

        n_rep = max(3, min(args.steps, 20))
        phase_ms = []
        for fn in (split_phase, combine_phase):
            fn()
            torch.cuda.synchronize()
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g, stream=stream):
                fn()
            for _ in range(2):
                g.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            for _ in range(n_rep):
                g.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            phase_ms.append(e0.elapsed_time(e1) / (n_rep * L))
            del g
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in order]
        call_ms = np.zeros(L)
        for rep in range(n_rep):
            q_static.copy_(qs[args.warmup + rep % args.steps])
            for j, layer in enumerate(order):
                ev[j][0].record(stream)
                cache.decode(layer, q_static[layer], out_static[layer], scale)
                ev[j][1].record(stream)
            torch.cuda.synchronize()
            for j, layer in enumerate(order):
                call_ms[layer] += ev[j][0].elapsed_time(ev[j][1]) / n_rep
    split_avg_ms, merge_avg_ms = phase_ms
    call_avg_ms = float(call_ms.mean())
    achieved = (bytes_step / L) / (split_avg_ms * 1e-3) / 1e9
    step_gbs = bytes_step / (step_ms * 1e-3) / 1e9
    tokens_per_s = w.batch / (step_ms * 1e-3)
    log(f"[bench] decode step {step_ms * 1e3:.1f} us -> {tokens_per_s:.1f} tok/s, {step_gbs:.0f} GB/s over the step; "
        f"split-K launch {split_avg_ms * 1e3:.2f} us -> {achieved:.0f} GB/s, combine {merge_avg_ms * 1e3:.2f} us, "
        f"one-call layer decode {call_avg_ms * 1e3:.2f} us")

    # ------------------------------------------------------------ prefill: probe + route + compress
    prefill = None
    if not args.no_prefill and w.batch == 1 and w.n_probe > 0:
        P = w.n_probe
        T = w.seq_lens[0]
        Qp = torch.empty((L, Hq, P, d), dtype=tdt, device=dev)
        for l in range(L):
            Qp[l].copy_(torch.from_numpy(gen.probe_queries(w, 0, layers=[l])[0]).to(dev).to(tdt))
        kl = [Ks[0][l] for l in range(L)]
        vl = [Vs[0][l] for l in range(L)]
        ql = [Qp[l] for l in range(L)]
        _, budget = B.layout(dm, [T], gen.fixed_modes(w, 0)[None])   # footprint of the 50/35/15 mix
        nbk = w.n_blocks
        ws = torch.empty(B.probe_workspace(dm, T, P), dtype=torch.uint8, device=dev)
        err = torch.empty((nbk, H, dm.n_err), dtype=torch.float32, device=dev)
        tscores = torch.empty((nbk, H, T), dtype=torch.float32, device=dev) if w.residual == 1 else None
        # per-token channel residuals: the probe's K selections, which compress reuses
        ksel = (torch.empty(B.selection_bytes(dm, T), dtype=torch.uint8, device=dev)
                if w.residual != 1 else None)
        _, all_exact = B.layout(dm, [T], np.full((1, nbk, H), 2, np.uint8))
        pcache_buf = torch.empty(all_exact, dtype=torch.uint8, device=dev)
        offs_dev = torch.empty((nbk, H), dtype=torch.int64, device=dev)
        modes_dev = torch.empty((nbk, H), dtype=torch.uint8, device=dev)
        times = {"probe": [], "route": [], "compress": [], "total": []}
        pmodes = None
        for rep in range(4):
            torch.cuda.synchronize()
            a0, a1, c0, c1 = (torch.cuda.Event(enable_timing=True) for _ in range(4))
            tw0 = time.perf_counter()
            a0.record()
            B.probe(dm, T, kl, ql, P, err, ws, None, tscores, ksel)
            a1.record()
            eh = err.cpu().numpy()                      # sync point
            tr0 = time.perf_counter()
            pmodes, lam, st = B.route(dm, T, eh, budget_bytes=budget, allow_infeasible=True)
            offs, total = B.layout(dm, [T], pmodes[None])
            tr1 = time.perf_counter()
            modes_dev.copy_(torch.from_numpy(pmodes))
            offs_dev.copy_(torch.from_numpy(offs[0].astype(np.int64)))
            c0.record()
            B.compress(dm, T, kl, vl, modes_dev, offs_dev, pcache_buf, None, tscores, ksel)
            c1.record()
            torch.cuda.synchronize()
            tw1 = time.perf_counter()
            if rep == 0:
                continue                                 # first pass warms up
            times["probe"].append(a0.elapsed_time(a1) * 1e-3)
            times["route"].append(tr1 - tr0)
            times["compress"].append(c0.elapsed_time(c1) * 1e-3)
            times["total"].append(tw1 - tw0)
        tp, trt, tc, tt = (float(np.mean(times[x])) for x in ("probe", "route", "compress", "total"))
        units = nbk * H
        usz = [nb for nb in w.block_sizes for _ in range(H)]
        cmp_read = T * 2 * d * e * L * H                                             # K and V of every layer
        cmp_write = sum(unit_read_bytes(w, int(m), T, nb) * (nb if (m & 3) == 2 else 1)
                        for m, nb in zip(pmodes.ravel(), usz))                # exact heads copy all nb layers
        # executed MFMA work of the deviation Gram kernels: per 16 tokens, 3 MFMAs (H H^T + H L^T + L H^T of
        # the bf16 hi/lo split) on each upper 32x32 tile of each matrix, 2 matrices per pair, 8 per block of four
        mfma_flops = sum(T * (d // 32) * (d // 32 + 1) // 2 * (2 if nb == 2 else 8) * 3 * (32 * 32 * 2) for nb in usz)
        if w.residual == 1:
            # token scores: every probe row of the block's layers against every token's deviation
            mfma_flops = sum(2 * nb * (Hq // H) * P * d * T for nb in usz)
        prefill = {
            "workload": "prefill8b" if w.name == "llama8b" else w.name,
            "probe_ms": tp * 1e3, "route_ms": trt * 1e3, "compress_ms": tc * 1e3,
            "wall_ms": tt * 1e3,
            "compressed_tokens_per_s": T / tt,
            "compress_gbs": (cmp_read + cmp_write) / tc / 1e9,
            "compress_frac_hbm": (cmp_read + cmp_write) / tc / 1e9 / HBM_PEAK_GBS,
            "probe_read_gbs": L * H * T * d * e / tp / 1e9,
            "probe_mfma_util": mfma_flops / tp / (MFMA_BF16_PEAK_TFLOPS * 1e12),
            "probe_mfma_tflop": mfma_flops / 1e12,
            "probe_mode_mix": np.bincount(pmodes.ravel() & 3, minlength=3).tolist(),
            "budget_bytes": int(budget), "lambda": lam,
        }
        if not args.no_cpu_baseline:
            prefill["cpu_baseline"] = cpu_baseline_prefill(w, pmodes.reshape(nbk, H), budget)
        log(f"[bench] prefill: probe {tp * 1e3:.2f} ms, route {trt * 1e3:.2f} ms, compress {tc * 1e3:.2f} ms "
            f"({prefill['compress_gbs']:.0f} GB/s), mix {prefill['probe_mode_mix']}")
        del Qp, ws, pcache_buf, tscores, ksel

    # ------------------------------------------------------------ generation: append + spans + tail, refresh
    generation = None
    if args.gen_tail > 0 and w.batch == 1 and w.n_probe > 0:
        from paper_2607_06519_amd.cache import Generation
        cap, Pr = args.gen_tail, min(w.n_probe, 64)
        g = Generation(dm, cache, cap)
        gq = torch.from_numpy(gen.decode_queries(w, 0)).to(dev).to(tdt)
        gk = torch.from_numpy(gen.decode_queries(w, 1)).to(dev).to(tdt)[:, :, :H].contiguous()  # stand-in K / V rows
        gv = torch.from_numpy(gen.decode_queries(w, 2)).to(dev).to(tdt)[:, :, :H].contiguous()
        gout = torch.empty_like(gq)
        rows = [torch.from_numpy(gen.probe_queries(w, 0, layers=[l])[0][:, :Pr]).to(dev).to(tdt)[None]
                for l in range(L)]

        def gstep():
            for layer in order:
                g.append(layer, gk[layer], gv[layer])
                g.decode(layer, gq[layer], gout[layer], scale)

        refresh_s = []
        for r in range(2):                      # two refreshes: the prefix plus two spans of `cap` tokens
            for _ in range(cap):
                gstep()
                g.advance()
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            g.refresh(rows, Pr, lam=float("inf"))
            torch.cuda.synchronize()
            refresh_s.append(time.perf_counter() - t0)
        for _ in range(cap // 2):               # the tail half full
            gstep()
            g.advance()
        gstream = torch.cuda.Stream()
        gstream.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(gstream):
            gstep()
            torch.cuda.synchronize()
            ggraph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(ggraph, stream=gstream):
                gstep()
            for _ in range(args.warmup):
                ggraph.replay()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(gstream)
            for _ in range(args.steps):
                ggraph.replay()
            e1.record(gstream)
            torch.cuda.synchronize()
        gen_ms = e0.elapsed_time(e1) / args.steps
        generation = {
            "tail_cap": cap, "spans": len(g.spans), "tail_rows": g.n_tail + 1,
            "context_tokens": w.max_seq_len + 2 * cap + g.n_tail + 1,
            "step_ms": gen_ms, "tokens_per_s": w.batch / (gen_ms * 1e-3),
            "refresh_ms": float(np.mean(refresh_s)) * 1e3,
            "refresh_ms_per_token": float(np.mean(refresh_s)) * 1e3 / cap,
            "note": "one step = for every layer an append into the exact tail and a decode over the "
                    "prefix span, two refreshed spans and the tail (graph replay); refresh = probe, route "
                    "(lambda = inf, all shared) and compress of the full tail, wall time",
        }
        log(f"[bench] generation: step {gen_ms * 1e3:.1f} us over {len(g.spans)} spans + tail, "
            f"refresh {generation['refresh_ms']:.2f} ms per {cap} tokens")
        del g

    # ------------------------------------------------------------ CPU oracle baseline
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(w, modes[0])

    traffic = load_traffic(w.name)
    cfg = {"workload": w.name, "n_layers": L, "n_kv_heads": H, "n_q_heads": Hq, "head_dim": d, "topk": k,
           "batch": w.batch, "seq_len": w.max_seq_len, "block_sizes": list(w.block_sizes),
           "mode_mix": np.bincount(modes.ravel() & 3, minlength=3).tolist(),
           "layer_order": args.order, "graph": graph is not None, "cache_gb": cache.total_bytes / 1e9,
           "bytes_per_step": bytes_step}
    if w.residual == 1:
        cfg["residual"] = "token set"
        if w.res_rates:
            rb = modes.ravel()[(modes.ravel() & 3) == 1] >> 2
            cfg["residual_fractions"] = [r / 1e6 for r in w.res_rates]
            cfg["residual_fraction_mix"] = np.bincount(rb, minlength=len(w.res_rates)).tolist()
        else:
            cfg["residual_fraction"] = w.res_ppm / 1e6
    res = {
        "metric": "compressed-KV decode attn tokens/s + achieved HBM GB/s vs 8 TB/s, 32k ctx",
        "value": tokens_per_s, "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": step_ms, "step_ms_stats": step_stats, "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype, "data": "synthetic (seeded generator, layers correlated along depth within each block, needles)",
        "config": cfg,
        "step_hbm_gbs": step_gbs,
        "roofline": {"bound": "hbm", "achieved": achieved, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": achieved / HBM_PEAK_GBS, "traffic": traffic,
                     "kernel": "decode_stream_kernel (the split-K launch of a layer, fdkv_decode_partial)",
                     "bytes_per_launch": bytes_step / L, "launch_us": split_avg_ms * 1e3,
                     "combine_us": merge_avg_ms * 1e3, "layer_call_us": call_avg_ms * 1e3,
                     "layer_call_frac": (bytes_step / L) / (call_avg_ms * 1e-3) / 1e9 / HBM_PEAK_GBS,
                     "step_frac": step_gbs / HBM_PEAK_GBS},
        "cpu_baseline": cpu,
        "prefill": prefill,
        "generation": generation,
    }
    if other:
        res["other_workloads"] = other
    print(json.dumps(res), flush=True)


def cpu_baseline_prefill(w, pmodes, budget):
    """The oracle's prefill (Eq. 2 probe in its literal form, budget route, compress) timed on a
    bounded sample of (block, KV head) units and scaled to the whole workload."""
    import numpy as np

    import oracle as O
    from synth import gen
    cores = len(os.sched_getaffinity(0))
    T, d, k, G = w.seq_lens[0], w.head_dim, w.topk, w.group
    units = [(b, h) for b in range(w.n_blocks) for h in range(w.n_kv_heads)]
    pick = []
    for m in (1, 0, 2):                       # up to three units of each mode the probe chose
        cand = [u for u in units if (int(pmodes[u]) & 3) == m]
        pick += cand[:3]
    probe_s, comp_s, E = [], {0: [], 1: [], 2: []}, []
    for (b, h) in pick:
        K, V, _ = gen.block_segment(w, 0, b, h)
        f, nb = w.blocks[b]
        Q = gen.probe_queries(w, 0, layers=list(range(f, f + nb)))[:, h * G:(h + 1) * G]
        t0 = time.perf_counter()
        E.append(O.routing_errors(K, Q, k))
        probe_s.append(time.perf_counter() - t0)
        m = int(pmodes[b, h]) & 3
        t0 = time.perf_counter()
        O.compress_unit(K, V, m, k, w.dtype)
        comp_s[m].append(time.perf_counter() - t0)
    # the budget search over every unit: the sampled losses, spread by seeded factors
    rng = np.random.default_rng(0)
    Eall = np.array([E[i % len(E)] for i in range(len(units))]) * rng.uniform(0.5, 1.5, (len(units), 1))
    t0 = time.perf_counter()
    O.route_budget(Eall, T, d, k, w.dtype, budget, [nb for nb in w.block_sizes for _ in range(w.n_kv_heads)])
    route_s = time.perf_counter() - t0
    counts = np.bincount(pmodes.ravel() & 3, minlength=3)
    t_probe = float(np.mean(probe_s)) * len(units)
    t_comp = float(sum(counts[m] * np.mean(comp_s[m]) for m in comp_s if comp_s[m]))
    total = t_probe + route_s + t_comp
    return {"value": T / total, "unit": "compressed tokens/s", "cores": cores, "kind": "oracle",
            "probe_s": t_probe, "route_s": route_s, "compress_s": t_comp,
            "sample": f"oracle Eq. 2 (literal logit matrices, fp64) on {len(pick)} (block, KV head) units "
                      f"({sum(probe_s):.1f}s) scaled to {len(units)}; compress of the same units "
                      f"({sum(sum(v) for v in comp_s.values()):.1f}s) scaled by the routed mix {counts.tolist()}; budget route "
                      f"over {len(units)} units ({route_s:.2f}s)"}


def cpu_baseline(w, modes):
    """The oracle's decode on a bounded sample: a few (block, KV head) units, all their layers, a few steps."""
    import numpy as np

    import oracle as O
    from synth import gen
    try:
        from threadpoolctl import threadpool_info
        blas_threads = max([i.get("num_threads", 1) for i in threadpool_info()] or [1])
    except Exception:  # pragma: no cover
        blas_threads = 1
    cores = len(os.sched_getaffinity(0))
    rng = np.random.default_rng(0)
    d, G = w.head_dim, w.group
    flat = [(b, h) for b in range(w.n_blocks) for h in range(w.n_kv_heads)]
    pick = []
    for m in (0, 1, 2):
        cand = [u for u in flat if (int(modes[u]) & 3) == m]
        pick += [cand[i] for i in rng.choice(len(cand), size=min(4, len(cand)), replace=False)]
    n_steps = 14                        # about 10 s of oracle work on the 8B shape
    elapsed, n_calls = 0.0, 0
    for (b, h) in pick:
        K, V, _ = gen.block_segment(w, 0, b, h)
        f, nb = w.blocks[b]
        m = int(modes[b, h]) & 3
        if w.residual == 1:
            tokens = None
            if m == 1:                  # the set the probe picks (selection is prefill work, not timed)
                QB = gen.probe_queries(w, 0, layers=list(range(f, f + nb)))[:, h * G:(h + 1) * G]
                sc, _ = O.token_scores(K, QB)
                tokens = O.residual_tokens(sc, O.n_residual_tokens(K.shape[1], unit_ppm(w, modes[b, h])))
            unit = O.compress_unit_tokens(K, V, m, tokens, w.dtype)
            dec = O.decode_unit_tokens
        else:
            unit = O.compress_unit(K, V, m, w.topk, w.dtype)
            dec = O.decode_unit
        for s in range(n_steps):
            q = gen.decode_queries(w, s)
            for layer in range(f, f + nb):
                qq = q[layer][0, h * G:(h + 1) * G].astype(np.float64)
                t0 = time.perf_counter()
                dec(unit, m, layer, qq, 1.0 / math.sqrt(d), d, nb)
                elapsed += time.perf_counter() - t0
                n_calls += 1
    per_unit_layer = elapsed / n_calls
    step_s = per_unit_layer * w.n_layers * w.n_kv_heads
    return {"value": w.batch / step_s, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "blas_threads": blas_threads,
            "sample": f"oracle decode (reconstruct + fp64 softmax attention) of {len(pick)} (block, KV head) units "
                      f"x their layers x {n_steps} steps = {n_calls} unit-layers ({elapsed:.1f}s), scaled to "
                      f"{w.n_layers * w.n_kv_heads} unit-layers per step"}


if __name__ == "__main__":
    main()
