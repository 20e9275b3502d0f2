#!/usr/bin/env python3
"""Throughput of the certified cache path on one MI355X.

One step = one pass of the whole path over one batch of B queries:
  spectral norm of the head (sync) -> lookup of the batch against the cache
  -> certification of the batch (labels, radii for write-back) -> insert of
  the misses (sync) -> the cache is rolled back to its N construction rows,
  so every step sees the same cache.
Inputs are resident in device memory before the timed region.  The cache is
built once beforehand (spectral norm, certification of N candidates, insert),
and that construction is timed and reported separately.

Prints ONE JSON line (rank 0): value = whole-step lookups/s; the fused lookup
kernel's roofline (HIP events on the stream the library launches on); and the
CPU oracle timed on a bounded sample on this host.

``--workload stream-d256-c200-bf16`` runs the streaming workload instead: 16
rounds (one step each) of lookup -> certify -> insert on a bfloat16 cache that
grows from 2,097,152 entries, reported per round and in aggregate.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"f16": 2500.0, "f32": 157.3}   # MI355X dense matrix peaks (fp16 = bf16 rate)
METRIC = "certified lookups/s and query·entry pairs/s at N=1M cache, d=256, C=200"


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def cpu_baseline(wl, zq_host, target_s: float):
    """The CPU oracle on a bounded sample of the same lookup.

    Main figure: ``oracle.lookup_blocked`` (float32 BLAS prefilter with a
    rigorous slack, float64 distances for the survivors; bit-identical to the
    plain definition) on every core the BLAS library uses.  Secondary: the
    plain definition ``oracle.lookup`` (float64 numpy, one thread).
    """
    import numpy as np

    import oracle
    t0 = time.perf_counter()
    sig = oracle.spectral_norm(wl.W).sigma
    cert = oracle.certify(wl.z, wl.W, wl.b, sig, store=wl.config.store_dtype)
    keep = cert.r > 0
    Z, R, Lb = cert.stored[keep], cert.r[keep], cert.label[keep]
    t_cert = time.perf_counter() - t0
    log(f"cpu oracle: certify of {wl.z.shape[0]} candidates in {t_cert:.1f} s")
    threads, blas = _blas_threads()

    def timed(fn, m, budget):
        rows = np.linspace(0, zq_host.shape[0] - 1, m).astype(np.int64)
        t0 = time.perf_counter()
        fn(zq_host[rows], Z, R, Lb)
        return time.perf_counter() - t0

    # blocked oracle: grow the sample until it takes a good share of the budget
    m, t = 64, 0.0
    while True:
        t = timed(oracle.lookup_blocked, m, target_s)
        if t > 0.4 * target_s or m >= zq_host.shape[0]:
            break
        m = int(min(zq_host.shape[0], max(2 * m, m * 0.6 * target_s / max(t, 1e-3))))
    log(f"cpu oracle (blocked, {threads} BLAS threads): {m} lookups in {t:.1f} s")
    t1 = timed(oracle.lookup, 1, 0)
    m1 = int(max(1, min(64, 0.25 * target_s / max(t1, 1e-6))))
    tp = timed(oracle.lookup, m1, 0)
    log(f"cpu oracle (plain definition, one thread): {m1} lookups in {tp:.1f} s")
    return {"value": m / t, "unit": "lookups/s", "cores": threads, "kind": "oracle",
            "sample": f"{m} queries of the batch, each against all {Z.shape[0]} entries with oracle.lookup_blocked "
                      f"({blas}, {threads} threads); pairs/s = {m * Z.shape[0] / t:.3e}",
            "seconds": t, "cpu_model": _cpu_model(), "certify_seconds": t_cert,
            "plain_definition": {"value": m1 / tp, "unit": "lookups/s", "cores": 1, "queries": m1,
                                 "seconds": tp, "function": "oracle.lookup (float64 numpy)"}}


def _blas_threads():
    try:
        from threadpoolctl import threadpool_info
        info = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if info:
            return int(info[0]["num_threads"]), f"{info[0]['internal_api']} {info[0].get('version', '')}".strip()
    except Exception:
        pass
    return len(os.sched_getaffinity(0)), "blas"


def measured_traffic(workload: str, precision: str):
    """HBM bytes per launch of the lookup kernel from the committed rocprofv3
    counter summary, or None when the kernel source changed since."""
    import hashlib
    path = os.path.join(ROOT, "profiles", f"lookup_{workload}_{precision}_counters.md")
    src = os.path.join(ROOT, "paper_2608_13144_amd", "csrc", "lookup.hip")
    try:
        with open(path) as f:
            line = next(l for l in f if l.startswith("traffic_json:"))
        rec = json.loads(line.split(":", 1)[1])
        with open(src, "rb") as f:
            sha = hashlib.sha256(f.read()).hexdigest()[:16]
    except (OSError, StopIteration, ValueError):
        return None
    if rec.get("lookup_hip_sha16") != sha:
        return None
    rec["file"] = os.path.basename(path)
    return rec


def _cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def stream_bench(args, cfg) -> int:
    """Streaming workload: rounds of lookup -> certify(B) -> insert(misses) on a
    growing cache.  The head is fixed, so sigma is computed once with the
    cache.  Each round's queries are composed on the host from the cache state
    at the start of the round (untimed); a round's timed region is the serve
    call (lookup, certify of the batch, insert with its one host sync)."""
    import numpy as np
    import torch

    from paper_2608_13144_amd import api
    from paper_2608_13144_amd import workload as wlmod

    dev = torch.device("cuda:0")
    N, B, d, C = cfg.n_cache, cfg.batch, cfg.d, cfg.C

    def g(x):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    t0 = time.perf_counter()
    wl = wlmod.make_workload(cfg, seed=0)
    log(f"workload {cfg.name}: N={N} B={B} d={d} C={C} rounds={cfg.rounds} drawn in {time.perf_counter() - t0:.1f} s")
    W, b, zc = g(wl.W), g(wl.b), g(wl.z)
    torch.cuda.synchronize()
    tc = time.perf_counter()
    sig = api.spectral_norm(W)
    cert = api.certify(zc, W, b, sig.sigma, store=cfg.store_dtype)
    cache = api.LipCache(d, cfg.cache_capacity, store=cfg.store_dtype, device=dev)
    cache.insert(zc, cert.label, cert.r)
    torch.cuda.synchronize()
    t_build = time.perf_counter() - tc
    del zc, cert
    log(f"cache built: n={cache.n} sigma={sig.sigma:.12f} in {t_build * 1e3:.1f} ms")

    def queries(t):
        draws = wlmod.draw_queries(wl, t)
        idx = torch.from_numpy(wlmod.near_indices(draws, cache.n)).to(dev)
        return wlmod.compose_queries(draws, cache.z[idx].float().cpu().numpy(), cache.r[idx].cpu().numpy())

    zq_host0 = queries(0)
    zq0 = g(zq_host0)
    for _ in range(args.warmup):      # lookups only: the cache is not touched
        cache.lookup(zq0, precision=args.precision, prune=args.prune)
    torch.cuda.synchronize()
    rounds, total_s, total_lk, flops = [], 0.0, 0.0, 0.0
    for t in range(cfg.rounds):
        zq = zq0 if t == 0 else g(queries(t))
        n_t = cache.n
        pruned_t = args.prune and cache.lookup_prunes(args.precision)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ts = time.perf_counter()
        e0.record()
        res = cache.lookup(zq, precision=args.precision, prune=args.prune)
        e1.record()
        cq = api.certify(zq, W, b, sig.sigma, store=cfg.store_dtype)
        ins = cache.insert(zq, cq.label, cq.r, res.label)
        torch.cuda.synchronize()
        dt = time.perf_counter() - ts
        lk = e0.elapsed_time(e1)
        hits = int(res.stats[0].item())
        rounds.append({"round": t, "n": n_t, "round_ms": dt * 1e3, "lookup_ms": lk, "hits": hits, "inserted": ins})
        total_s += dt
        total_lk += lk * 1e-3
        flops += 2.0 * B * n_t * (32 if pruned_t else d)
        log(f"round {t}: n={n_t} round {dt * 1e3:.2f} ms lookup {lk:.2f} ms hits {hits}/{B} inserted {ins}")
    achieved = flops / total_lk / 1e12
    peak = PEAK_TFLOPS[args.precision]
    pairs = sum(B * r["n"] for r in rounds)
    out = {
        "metric": METRIC,
        "value": B * cfg.rounds / total_s,
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": cfg.rounds,
        "warmup": args.warmup,
        "ms_per_step": total_s / cfg.rounds * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.precision,
        "data": "synthetic",
        "config": {"workload": cfg.name, "N": N, "B": B, "d": d, "C": C, "store": cfg.store_dtype,
                   "rounds": cfg.rounds, "precision": args.precision,
                   "step": "one round: lookup+certify(B)+insert(misses)",
                   "lookup": "pruned (LIPCACHE_LOOKUP_PRUNE)" if args.prune else "full"},
        "pairs_per_s": pairs / total_s,
        "lookup_pairs_per_s": pairs / total_lk,
        "final_n": cache.n,
        "cache_build_ms": t_build * 1e3,
        "rounds": rounds,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": None,
                     "kernel": "lookup_dma_kernel (fused contraction + filter + re-check)",
                     "algorithmic": (f"sum over rounds of 2*B*n_t*d = {flops:.4e} flop" if not args.prune else
                                     f"sum over rounds of the prefix contraction 2*B*n_t*32 = {flops:.4e} flop "
                                     "(pruned lookup)")},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, zq_host0, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


def construct_bench(args, cfg) -> int:
    """Offline construction (Alg. 1) of a cache from the workload's N candidates:
    spectral norm, certify with the tight radius (the paper's default),
    select with the chosen strategy under a per-class budget.  One step =
    the whole construction into an emptied cache."""
    import numpy as np
    import torch

    from paper_2608_13144_amd import api
    from paper_2608_13144_amd import workload as wlmod

    dev = torch.device("cuda:0")
    N, d, C = cfg.n_cache, cfg.d, cfg.C
    t0 = time.perf_counter()
    wl = wlmod.make_workload(cfg, seed=0)
    log(f"workload {cfg.name}: {N} candidates, d={d}, C={C}; drawn in {time.perf_counter() - t0:.1f} s")
    g = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)  # noqa: E731
    W, b, z = g(wl.W), g(wl.b), g(wl.z)
    budget = args.per_class * C
    cache = api.LipCache(d, budget, store=cfg.store_dtype, device=dev)
    pri = g(np.random.default_rng(1).random(N).astype(np.float32)) if args.construct == "priority" else None

    def step():
        cache.n = 0
        s = api.spectral_norm(W).sigma
        cert = api.certify(z, W, b, s, store=cfg.store_dtype, radius_mode="tight")
        return cache.construct(z, cert.label, cert.r, strategy=args.construct, per_class=args.per_class,
                               n_classes=C, priority=pri)

    for _ in range(max(1, args.warmup)):
        step()
    torch.cuda.synchronize()
    times = []
    for _ in range(args.steps):
        ts = time.perf_counter()
        n_app, _sel = step()
        torch.cuda.synchronize()
        times.append(time.perf_counter() - ts)
    t = float(np.median(times))
    log(f"construct {args.construct}: {n_app} of {N} candidates appended; median {t * 1e3:.2f} ms per construction")
    out = {
        "metric": "offline construction (Alg. 1): candidates processed per second",
        "value": N / t,
        "unit": "candidates/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": t * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": cfg.name, "N": N, "d": d, "C": C, "strategy": args.construct,
                   "per_class": args.per_class, "radius": "tight",
                   "step": "spectral_norm+certify(N, tight)+construct"},
        "appended": n_app,
        "roofline": None,
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline:
        import oracle
        m = min(N, 4000)
        ts = time.perf_counter()
        sig = oracle.spectral_norm(wl.W).sigma
        cert = oracle.certify(wl.z[:m], wl.W, wl.b, sig, store=cfg.store_dtype, radius_mode="tight")
        st = oracle.CacheState(d=d, capacity=budget, store=cfg.store_dtype)
        oracle.construct(st, wl.z[:m], cert.label, cert.r, strategy=args.construct, budget_per_class=args.per_class,
                         n_classes=C, priority=None if pri is None else pri.cpu().numpy()[:m])
        tc = time.perf_counter() - ts
        out["cpu_baseline"] = {"value": m / tc, "unit": "candidates/s", "cores": _blas_threads()[0], "kind": "oracle",
                               "sample": f"the first {m} candidates (tight certify + oracle.construct)",
                               "seconds": tc}
    print(json.dumps(out), flush=True)
    return 0


def boundaries_bench(args, cfg) -> int:
    """The reuse-boundary comparison of the paper's Sec. 6 on a synthetic workload:
    for each boundary, the hit rate, the certified-consistency rate (hits
    returning the head's own argmax at the query) and the lookup time."""
    import numpy as np
    import torch

    from paper_2608_13144_amd import api
    from paper_2608_13144_amd import workload as wlmod

    dev = torch.device("cuda:0")
    N, B, d, C = cfg.n_cache, cfg.batch, cfg.d, cfg.C
    wl = wlmod.make_workload(cfg, seed=0)
    g = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)  # noqa: E731
    W, b, zc = g(wl.W), g(wl.b), g(wl.z)
    sig = api.spectral_norm(W).sigma
    cert = api.certify(zc, W, b, sig, store=cfg.store_dtype)
    tight = api.certify(zc, W, b, sig, store=cfg.store_dtype, radius_mode="tight")
    cache = api.LipCache(d, N, store=cfg.store_dtype, device=dev)
    cache.insert(zc, cert.label, cert.r)
    draws = wlmod.draw_queries(wl, 0)
    idx = torch.from_numpy(wlmod.near_indices(draws, cache.n)).to(dev)
    zq = g(wlmod.compose_queries(draws, cache.z[idx].float().cpu().numpy(), cache.r[idx].cpu().numpy()))
    head = api.certify(zq, W, b, sig, store=cfg.store_dtype).label
    r_med = float(cache.r[: cache.n].median().item())
    boundaries = [("certified conservative (Eq. 21)", cache.r[: cache.n]),
                  ("certified tight (Remark 5.1)", tight.r[: cache.n]),
                  ("tightened 0.5 x conservative", cache.boundary_radius("scaled", 0.5)),
                  (f"global threshold tau = 2 x median r = {2 * r_med:.4f}", cache.boundary_radius("global", 2 * r_med)),
                  ("inter-class empirical (half the nearest class-mean gap)",
                   cache.boundary_radius("interclass", 1.0, n_classes=C))]
    rows = []
    for name, r in boundaries:
        view = cache.with_radii(r.contiguous())
        for _ in range(max(1, args.warmup)):
            res = view.lookup(zq)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            res = view.lookup(zq)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        hits, cons = api.consistency(res.label, head)
        rows.append({"boundary": name, "hit_rate": hits / B, "consistency_rate": (cons / hits) if hits else None,
                     "hits": hits, "consistent": cons, "lookup_ms": ms,
                     "rechecked_pairs": int(res.stats[1].item())})
        log(f"{name}: hit rate {hits / B:.4f}, consistency {cons}/{hits}, lookup {ms:.2f} ms")
    out = {
        "metric": "reuse boundaries: hit rate and certified-consistency rate",
        "value": B / (rows[0]["lookup_ms"] * 1e-3),
        "unit": "lookups/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": rows[0]["lookup_ms"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": args.precision, "data": "synthetic",
        "config": {"workload": cfg.name, "N": N, "B": B, "d": d, "C": C, "step": "lookup per boundary"},
        "boundaries": rows,
        "roofline": None, "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)
    return 0


def indexed_bench(args, cfg) -> int:
    """The exact cluster-pruned lookup (an index of K clusters over the cache)
    against the dense lookup on the same cache and batch: one step = one
    indexed lookup of the batch (query plan, pruned scan, finalize; one
    host read-back).  The index build is timed once and reported."""
    import numpy as np
    import torch

    from paper_2608_13144_amd import api
    from paper_2608_13144_amd import workload as wlmod

    dev = torch.device("cuda:0")
    N, B, d, C = cfg.n_cache, cfg.batch, cfg.d, cfg.C
    wl = wlmod.make_workload(cfg, seed=0)
    g = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)  # noqa: E731
    W, b, zc = g(wl.W), g(wl.b), g(wl.z)
    sig = api.spectral_norm(W).sigma
    cert = api.certify(zc, W, b, sig, store=cfg.store_dtype)
    cache = api.LipCache(d, N, store=cfg.store_dtype, device=dev)
    cache.insert(zc, cert.label, cert.r)
    draws = wlmod.draw_queries(wl, 0)
    idx = torch.from_numpy(wlmod.near_indices(draws, cache.n)).to(dev)
    zq = g(wlmod.compose_queries(draws, cache.z[idx].float().cpu().numpy(), cache.r[idx].cpu().numpy()))
    K = args.indexed
    ix = cache.build_index(K, args.index_iters)  # warm-up build
    torch.cuda.synchronize()
    tb = time.perf_counter()
    ix = cache.build_index(K, args.index_iters)
    torch.cuda.synchronize()
    build_ms = (time.perf_counter() - tb) * 1e3
    sizes = np.diff(ix.offsets.cpu().numpy())
    log(f"index K={K} iters={args.index_iters}: built in {build_ms:.1f} ms; cluster sizes "
        f"min {sizes.min()} median {int(np.median(sizes))} max {sizes.max()}; "
        f"dead {int((ix.bound.cpu().numpy() == -np.inf).sum())}")
    for _ in range(max(1, args.warmup)):
        res_d = cache.lookup(zq, precision=args.precision)
        res_i, pairs = cache.lookup_indexed(ix, zq, precision=args.precision)
    torch.cuda.synchronize()
    same = bool(torch.equal(res_i.label, res_d.label) and torch.equal(res_i.index, res_d.index))
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(args.steps):
        cache.lookup(zq, precision=args.precision, out=res_d)
    e1.record()
    torch.cuda.synchronize()
    dense_ms = e0.elapsed_time(e1) / args.steps
    t0 = time.perf_counter()
    for _ in range(args.steps):
        res_i, pairs = cache.lookup_indexed(ix, zq, precision=args.precision, out=res_i)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) / args.steps * 1e3
    frac = pairs / (B * cache.n)
    log(f"indexed lookup {ms:.3f} ms vs dense {dense_ms:.3f} ms ({dense_ms / ms:.1f}x); pairs scanned "
        f"{pairs} = {frac:.4f} of B*N; same answers as dense: {same}")
    flops = 2.0 * pairs * d
    achieved = flops / (ms * 1e-3) / 1e12
    peak = PEAK_TFLOPS[args.precision]
    out = {
        "metric": "indexed certified lookups per second (exact cluster-pruned lookup)",
        "value": B / (ms * 1e-3),
        "unit": "lookups/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": args.precision, "data": "synthetic",
        "config": {"workload": cfg.name, "N": cache.n, "B": B, "d": d, "C": C, "K": K,
                   "index_iters": args.index_iters, "step": "lookup_indexed (plan + pruned scan + finalize)"},
        "dense_lookup_ms": dense_ms,
        "speedup_vs_dense": dense_ms / ms,
        "pairs_scanned": pairs,
        "pairs_fraction": frac,
        "index_build_ms": build_ms,
        "same_answers_as_dense": same,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": None,
                     "kernel": "whole indexed lookup (plan + scan + finalize)",
                     "algorithmic": f"2*pairs*d = {flops:.4e} flop per lookup"},
        "cpu_baseline": None,
    }
    print(json.dumps(out), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.splitlines()[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="mix-d256-c200")
    ap.add_argument("--precision", default="f16", choices=["f16", "f32"])
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="target oracle time for cpu_baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--construct", default="", choices=["", "radius_dedup", "priority", "kcenter"],
                    help="time the offline construction (Alg. 1) of a cache from the workload's candidates")
    ap.add_argument("--per-class", type=int, default=200, help="per-class budget of --construct")
    ap.add_argument("--indexed", type=int, default=0, metavar="K",
                    help="time the exact cluster-pruned lookup with K clusters against the dense lookup")
    ap.add_argument("--index-iters", type=int, default=4, help="Lloyd iterations of the index build")
    ap.add_argument("--index-k", type=int, default=256, metavar="K",
                    help="also run the batch through a K-cluster index after the timed steps (0: skip)")
    ap.add_argument("--prune", action="store_true",
                    help="time the step with the pruned lookup (LIPCACHE_LOOKUP_PRUNE; same answers)")
    ap.add_argument("--no-prune-context", action="store_true",
                    help="skip timing the pruned lookup of the batch after the timed steps")
    ap.add_argument("--boundaries", action="store_true",
                    help="compare reuse boundaries (hit rate, certified-consistency rate) on the workload")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (5 times) to calibrate HBM byte counters")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(the lookup would shard by queries or by cache rows; see DESIGN.md)", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration_bytes_read": n * 4, "copy_calibration_bytes_written": n * 4,
                          "launches": 5}), flush=True)
        return 0

    from paper_2608_13144_amd import api
    from paper_2608_13144_amd import workload as wlmod

    dev = torch.device("cuda:0")
    cfg = wlmod.CONFIGS[args.workload]
    if args.construct:
        return construct_bench(args, cfg)
    if args.boundaries:
        return boundaries_bench(args, cfg)
    if args.indexed:
        return indexed_bench(args, cfg)
    if cfg.rounds != 1:
        return stream_bench(args, cfg)
    N, B, d, C = cfg.n_cache, cfg.batch, cfg.d, cfg.C

    def g(x):
        return torch.from_numpy(np.ascontiguousarray(x)).to(dev)

    t0 = time.perf_counter()
    wl = wlmod.make_workload(cfg, seed=0)
    log(f"workload {cfg.name}: N={N} B={B} d={d} C={C} drawn in {time.perf_counter() - t0:.1f} s")
    W, b, zc = g(wl.W), g(wl.b), g(wl.z)

    # ---- cache construction (untimed here, reported)
    torch.cuda.synchronize()
    tc = time.perf_counter()
    sig = api.spectral_norm(W)
    cert = api.certify(zc, W, b, sig.sigma, store=cfg.store_dtype)
    cache = api.LipCache(d, N + B, store=cfg.store_dtype, device=dev)
    cache.insert(zc, cert.label, cert.r)
    torch.cuda.synchronize()
    t_build = time.perf_counter() - tc
    n0 = cache.n
    log(f"cache built: n={n0} sigma={sig.sigma:.12f} ({sig.iterations} iterations) in {t_build * 1e3:.1f} ms")

    draws = wlmod.draw_queries(wl, 0)
    idx = wlmod.near_indices(draws, n0)
    it = torch.from_numpy(idx).to(dev)
    centres = cache.z[it].float().cpu().numpy()
    radii = cache.r[it].cpu().numpy()
    zq_host = wlmod.compose_queries(draws, centres, radii)
    zq = g(zq_host)
    res = api.LookupResult(torch.empty(B, dtype=torch.int32, device=dev),
                           torch.empty(B, dtype=torch.int64, device=dev),
                           torch.empty(B, dtype=torch.float32, device=dev),
                           torch.zeros(4, dtype=torch.int64, device=dev),
                           torch.empty(B, dtype=torch.uint8, device=dev))
    # events per step: 0 before lookup, 1 after lookup, 2 after sigma, 3 after certify, 4 after insert.
    # The lookup does not need sigma, so it is issued first: the synchronous
    # spectral-norm call's host-side launches then overlap the scan.
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(5)] for _ in range(args.steps)]
    inserted = []

    def step(i: int | None):
        if i is not None:
            ev[i][0].record()
        cache.lookup(zq, precision=args.precision, out=res, prune=args.prune)
        if i is not None:
            ev[i][1].record()
        s = api.spectral_norm(W).sigma
        if i is not None:
            ev[i][2].record()
        cq = api.certify(zq, W, b, s, store=cfg.store_dtype)
        if i is not None:
            ev[i][3].record()
        inserted.append(cache.insert(zq, cq.label, cq.r, res.label))
        if i is not None:
            ev[i][4].record()
        cache.n = n0

    for _ in range(args.warmup):
        step(None)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(args.steps):
        step(i)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    parts = np.array([[e[j].elapsed_time(e[j + 1]) for j in range(4)] for e in ev])
    lk_ms = parts[:, 0].tolist()
    lk = sum(lk_ms) / len(lk_ms)
    comp = {"spectral_norm_ms": float(parts[:, 1].mean()), "lookup_ms": lk,
            "lookup_median_ms": float(np.median(parts[:, 0])), "certify_batch_ms": float(parts[:, 2].mean()),
            "insert_ms": float(parts[:, 3].mean())}
    log("per step: " + ", ".join(f"{k} {v:.3f}" for k, v in comp.items()))
    stats = res.stats.cpu().tolist()
    hits = int(stats[0])
    log(f"{args.steps} steps in {elapsed:.3f} s; lookup {lk:.3f} ms avg (min {min(lk_ms):.3f}); "
        f"hits {hits}/{B}; rechecked {stats[1]}; band pairs {stats[2]}; inserted/step {inserted[-1]}")

    pruned_path = args.prune and cache.lookup_prunes(args.precision)
    flops = 2.0 * B * n0 * d
    if pruned_path:
        # the matrix work every pair gets: the first 32 features (blocks the
        # prefix filter keeps also run the rest of the contraction)
        flops = 2.0 * B * n0 * 32
    achieved = flops / (lk * 1e-3) / 1e12
    peak = PEAK_TFLOPS[args.precision]
    out = {
        "metric": METRIC,
        "value": B * args.steps / elapsed,
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": elapsed / args.steps * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": args.precision,
        "data": "synthetic",
        "config": {"workload": cfg.name, "N": n0, "B": B, "d": d, "C": C, "store": cfg.store_dtype,
                   "precision": args.precision, "step": "spectral_norm+lookup+certify(B)+insert(misses)"},
        "pairs_per_s": B * n0 * args.steps / elapsed,
        "lookup_ms": lk,
        "components_ms": comp,
        "lookup_lookups_per_s": B / (lk * 1e-3),
        "lookup_pairs_per_s": B * n0 / (lk * 1e-3),
        "hit_rate": hits / B,
        "cache_build_ms": t_build * 1e3,
        "roofline": {"bound": "mfma", "achieved": achieved, "peak": peak, "unit": "TFLOP/s",
                     "frac": achieved / peak, "traffic": None,
                     "kernel": "lookup_dma_kernel (fused contraction + filter + re-check)",
                     "algorithmic": (f"2*B*N*d = {flops:.4e} flop per launch" if not pruned_path else
                                     f"prefix contraction 2*B*N*32 = {flops:.4e} flop per launch (pruned lookup)")},
        "cpu_baseline": None,
    }
    tr = measured_traffic(cfg.name, args.precision)
    if tr is not None and n0 == N:
        out["roofline"]["traffic"] = tr["traffic_bytes"]
        out["roofline"]["traffic_unit"] = "bytes per launch (FETCH_SIZE x %.4f + WRITE_SIZE x %.4f)" % (
            tr["fetch_scale"], tr["write_scale"])
        out["roofline"]["traffic_source"] = ("committed counter profile profiles/%s (rocprofv3 --pmc, taken on the "
                                             "lookup.hip with sha256 prefix %s, which this run also uses); not "
                                             "measured in this run" % (tr["file"], tr["lookup_hip_sha16"]))
        out["roofline"]["hbm_gbs"] = tr["traffic_bytes"] / (lk * 1e-3) / 1e9
    else:
        out["roofline"]["traffic_source"] = "none: no counter profile of the current lookup.hip is committed"
    if args.prune:
        out["config"]["lookup"] = ("pruned (LIPCACHE_LOOKUP_PRUNE)" if pruned_path else
                                   "LIPCACHE_LOOKUP_PRUNE requested; this cache takes the full path")
    elif not args.no_prune_context:
        try:
            out["pruned_lookup"] = pruned_context(cache, zq, res, lk, args)
        except Exception as e:  # context only: report it, keep the headline line
            log(f"pruned lookup context failed: {e}")
            out["pruned_lookup"] = {"error": str(e)}
    if args.index_k > 0:
        try:
            out["indexed_lookup"] = indexed_context(cache, zq, res, args)
        except Exception as e:  # context only: report it, keep the headline line
            log(f"indexed lookup context failed: {e}")
            out["indexed_lookup"] = {"K": args.index_k, "error": str(e)}
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, zq_host, args.cpu_seconds)
    print(json.dumps(out), flush=True)
    return 0


def pruned_context(cache, zq, res, full_ms, args) -> dict:
    """The same batch through the pruned lookup (LIPCACHE_LOOKUP_PRUNE; outside
    the timed steps): HIP-event time of the call and whether every answer
    equals the full lookup's.  Context for the headline, which stays the full
    contraction of every pair."""
    import numpy as np
    import torch

    out_p = cache.lookup(zq, precision=args.precision, prune=True)
    torch.cuda.synchronize()
    same = all(torch.equal(getattr(res, f).view(torch.uint8), getattr(out_p, f).view(torch.uint8))
               for f in ("label", "index", "dist2", "band"))
    sf, sp = res.stats.cpu().tolist(), out_p.stats.cpu().tolist()
    same = same and sf[0] == sp[0] and sf[2] == sp[2] and sf[3] == sp[3]
    ts = []
    for _ in range(10):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        cache.lookup(zq, precision=args.precision, out=out_p, prune=True)
        e1.record()
        torch.cuda.synchronize()
        ts.append(e0.elapsed_time(e1))
    ms = float(np.median(ts))
    B = zq.shape[0]
    log(f"pruned lookup: {ms:.3f} ms ({full_ms / ms:.2f}x the full lookup), same answers: {same}, "
        f"re-checked pairs {sp[1]} (full {sf[1]})")
    return {"lookup_ms": ms, "lookups_per_s": B / (ms * 1e-3), "pairs_per_s": B * cache.n / (ms * 1e-3),
            "speedup_vs_full_lookup": full_ms / ms, "same_answers_as_full": bool(same),
            "rechecked_pairs": int(sp[1]), "rechecked_pairs_full": int(sf[1])}


def indexed_context(cache, zq, res, args) -> dict:
    """The same batch through the exact cluster index (outside the timed
    steps): build time, lookup time and whether the answers equal the dense
    lookup's.  Context for the headline, which stays the dense scan."""
    import numpy as np
    import torch

    ix = cache.build_index(args.index_k, 4)
    torch.cuda.synchronize()
    tb = time.perf_counter()
    ix = cache.build_index(args.index_k, 4)
    torch.cuda.synchronize()
    build_ms = (time.perf_counter() - tb) * 1e3
    out_i, pairs = cache.lookup_indexed(ix, zq, precision=args.precision)
    same = bool(torch.equal(out_i.label, res.label) and torch.equal(out_i.index, res.index))
    ts = []
    for _ in range(5):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        cache.lookup_indexed(ix, zq, precision=args.precision, out=out_i)
        torch.cuda.synchronize()
        ts.append((time.perf_counter() - t0) * 1e3)
    ms = float(np.median(ts))
    B = zq.shape[0]
    log(f"indexed lookup (K={args.index_k}): {ms:.3f} ms, {pairs / (B * cache.n):.4f} of the pairs, "
        f"same answers as the dense lookup: {same}")
    return {"K": args.index_k, "build_ms": build_ms, "lookup_ms": ms, "lookups_per_s": B / (ms * 1e-3),
            "pairs_fraction": pairs / (B * cache.n), "same_answers_as_dense": same}


if __name__ == "__main__":
    sys.exit(main())
