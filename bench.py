"""Throughput of the cached mixed-precision EmbeddingBag training step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config industrial] [--gpus 1]

One step = forward (tag probe, gather + dequantize, sum-pool) + backward_update
(sort/de-dup, merged gradients, priority update, replacement, optimizer, write-back,
evict/fill) over one batch of synthetic Zipf-skewed lookups already resident in
HBM.  Prints one JSON line: pooled lookups/s (value), algorithmic HBM GB/s and its
fraction of peak for the whole step, the roofline of the dominant kernel, median /
p90 and cold-cache step times, a measured device copy bandwidth, and the CPU oracle
timed on a bounded sample with threads over tables.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from paper_2010_11305_amd import configs, workload  # noqa: E402

METRIC = "pooled lookups/sec + achieved HBM GB/s (fwd+bwd+update), 1 MI355X"
HBM_PEAK_GBS = 8000.0
COUNTERS_FILE = os.path.join(ROOT, "profiles", "industrial_step_hbm_counters.md")
# sources that determine the row-update kernel's code (its HBM counters go stale when they change)
UPDATE_KERNEL_SOURCES = ["k_update.hip", "embc_device.h", "embc_internal.h", "embc_dispatch.h", "embc_sort.h"]


def update_kernel_digest():
    import hashlib
    h = hashlib.sha256()
    for f in UPDATE_KERNEL_SOURCES:
        with open(os.path.join(ROOT, "paper_2010_11305_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_update_traffic():
    """HBM bytes per k_update launch from the committed counter summary (reads from the L2's
    requests to the memory fabric by size, writes from WRITE_SIZE; that file gives the
    commands and the calibration), or None when the summary was taken on other kernel
    sources."""
    try:
        text = open(COUNTERS_FILE).read()
    except OSError:
        return None
    vals = dict(line.split(":", 1) for line in text.splitlines() if line.startswith("k_update_"))
    try:
        if vals["k_update_source_digest"].strip() != update_kernel_digest():
            return None
        return float(vals["k_update_hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def record_bytes(cfg):
    """rho: bytes of one row of the low-precision table (codes + (s,b), or FP16 elements)."""
    if cfg["bits"] == 16:
        return 2 * cfg["dim"]
    return cfg["dim"] * cfg["bits"] // 8 + (4 if cfg["sb_fp16"] else 8)


def describe(cfg):
    T, N = len(cfg["rows"]), cfg["rows"][0]
    pool = cfg["pooling"]
    prec = "FP16" if cfg["bits"] == 16 else f"INT{cfg['bits']} + {'FP16' if cfg['sb_fp16'] else 'FP32'} (s,b)"
    return (f"{cfg['name']}: {T} tables x {N} rows x d{cfg['dim']} {prec}; FP32 cache {cfg['cache_fraction']:.0%} "
            f"{cfg['assoc']}-way {cfg['policy'].upper()}; B={cfg['batch']} bags/table, pooling {pool}; "
            f"Zipf {cfg['zipf']}; {cfg['optimizer']} lr {cfg['lr']}; {cfg['rounding']} rounding")


def algorithmic_bytes(cfg, st, B, decay_step=False):
    """Bytes the method must move for one table and one step (each unique row once).

    Forward:  4L + 4(B+1) indices/offsets, 4*assoc*U tag probes, 4d*U_h cached rows,
              rho*U_m low-precision rows, 4dB pooled output.
    Backward: 4L + 4(B+1), 4dB output gradients, row re-read (4d*U_h + rho*U_m),
              row writes (4d*(U_h - E_h) + rho*(E_h + U_byp) + 4d*U_ins), displaced
              residents V_o*(4d + rho), tags + stamps of inserts (8 U_ins) and stamps
              of hits (4 U_h, LRU), Adagrad (8 U), LFU counts (8 U, + 8N on decay steps).
    """
    d = cfg["dim"]
    phi = 4 * d
    rho = record_bytes(cfg)
    L, U, Uh = st["bwd_lookups"], st["unique"], st["unique_hits"]
    Um = U - Uh
    Eh, Ubyp, Uins = st["hit_evictions"], st["bypasses"], st["inserts"]
    Vo = st["evictions"] - Eh
    A = cfg["assoc"]
    fwd = 4 * L + 4 * (B + 1) + 4 * A * U + phi * Uh + rho * Um + 4 * d * B
    bwd = 4 * L + 4 * (B + 1) + 4 * d * B + phi * Uh + rho * Um
    bwd += phi * (Uh - Eh) + rho * (Eh + Ubyp) + phi * Uins + Vo * (phi + rho) + 8 * Uins
    if cfg["policy"] == "lru":
        bwd += 4 * Uh
    else:
        bwd += 8 * U
    if cfg["optimizer"] == "adagrad":
        bwd += 8 * U
    return fwd, bwd


def update_kernel_bytes(cfg, st):
    """Algorithmic bytes of the row-update kernel (k_update) for one table and one step,
    counting only the per-step terms of the method (each unique row once).

    It handles every unique row except the residents displaced after their own update
    (E_h, handled with the evictions): it re-reads the row (phi from the cache for a
    hit, rho from T for a miss), writes it to its way (phi: hit or insert) or to T
    (rho: bypass), writes the tag and LRU stamp of an insert (8; the tag alone, 4,
    under LFU), and reads and writes the Adagrad accumulator (8).  The output
    gradients are counted once per step (4dB) and not here; what the kernel reads to
    form each merged gradient is implementation cost (merged_gradient_bytes).
    """
    d = cfg["dim"]
    phi = 4 * d
    rho = record_bytes(cfg)
    U, Uh, Eh = st["unique"], st["unique_hits"], st["hit_evictions"]
    Uins, Ubyp = st["inserts"], st["bypasses"]
    rows = U - Eh
    b = phi * (Uh - Eh) + rho * (Uins + Ubyp)                           # row re-read
    b += phi * (Uh - Eh) + phi * Uins + rho * Ubyp                     # row writes
    b += (8 if cfg["policy"] == "lru" else 4) * Uins                   # tag (+ stamp) of inserts
    if cfg["optimizer"] == "adagrad":
        b += 8 * rows                                                  # accumulator read + write
    return b


def merged_gradient_bytes(cfg, st):
    """One FP32 merged-gradient row per row k_update handles: the least the kernel reads
    to apply the optimizer (implementation cost, not algorithmic bytes)."""
    return 4 * cfg["dim"] * (st["unique"] - st["hit_evictions"])


def host_description():
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    mem_gb = None
    try:
        with open("/proc/meminfo") as f:
            for line in f:
                if line.startswith("MemTotal"):
                    mem_gb = round(int(line.split()[1]) / 2**20, 1)
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except AttributeError:
        avail = os.cpu_count()
    return {"nproc": avail, "cpu_model": model, "mem_gib": mem_gb}


def _oracle_table_run(cfg, t, steps, budget_s, out, slot):
    """The oracle on table t alone (its own instance), fed that table's stream and
    gradients; forward + backward_update per step until the budget is spent."""
    import oracle  # test infrastructure: only this leg of the benchmark loads it

    one = dict(cfg, rows=[cfg["rows"][t]])
    o = oracle.Oracle(one["rows"], one["dim"], one["bits"], one["sb_fp16"], one["cache_fraction"], one["assoc"],
                      one["policy"], one.get("lfu_decay_interval", 0), one["rounding"] == "stochastic",
                      one["optimizer"] == "adagrad", one["lr"], one["eps"], one["seed"])
    o.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    B = cfg["batch"]
    sampler = workload.ZipfSampler(cfg["rows"][t], cfg["zipf"])
    lookups, elapsed, done = 0, 0.0, 0
    for k in range(steps):
        lengths = workload.bag_lengths(cfg, k, t)
        off = np.zeros(B + 1, dtype=np.int64)
        np.cumsum(lengths, out=off[1:])
        idx = workload.table_indices(cfg, k, t, int(off[-1]), sampler)
        off = off.astype(np.int32)
        g = workload._rng(cfg["grad_seed"], k, 99, t).standard_normal((B, 1, cfg["dim"]), dtype=np.float32)
        g *= np.float32(cfg["grad_sigma"])
        t0 = time.perf_counter()
        o.forward(idx, off, B)
        o.backward_update(idx, off, B, g)
        elapsed += time.perf_counter() - t0
        lookups += int(off[-1])
        done += 1
        if elapsed > budget_s:
            break
    out[slot] = (lookups, elapsed, done)


def cpu_baseline(cfg, steps, budget_s, threads, max_rows=0):
    """The CPU oracle, threads over tables (tables are independent): thread i runs table
    i alone; the rate is the sum of lookups over the slowest thread's oracle time.  With
    max_rows, each table is cut to that many rows (a row-scaled slice of the same batch
    shape, for tables too large for the host's memory or time)."""
    import threading

    full = cfg
    if max_rows:
        cfg = dict(cfg, rows=[min(int(r), int(max_rows)) for r in cfg["rows"]])
    T = len(cfg["rows"])
    n = max(1, min(threads, T))
    res = [None] * n
    th = [threading.Thread(target=_oracle_table_run, args=(cfg, i, steps, budget_s, res, i)) for i in range(n)]
    for x in th:
        x.start()
    for x in th:
        x.join()
    lookups = sum(r[0] for r in res)
    wall = max(r[1] for r in res)
    one = res[0][0] / res[0][1]
    desc = host_description()
    sliced = f" (row-scaled slice: {cfg['rows'][0]} of {full['rows'][0]} rows)" if cfg["rows"] != full["rows"] else ""
    sample = (f"tables 0..{n - 1} of {T} ({cfg['rows'][0]} rows each{sliced}), one oracle instance and one thread per "
              f"table, {min(r[2] for r in res)}-{max(r[2] for r in res)} steps of fwd+bwd+update each, "
              f"{lookups} lookups; the rate is per lookup of this {n}-table slice (tables are independent, so the "
              f"whole workload runs at the same rate per lookup); host: {desc['nproc']} usable cores, "
              f"{desc['cpu_model']}, {desc['mem_gib']} GiB")
    return {"value": lookups / wall, "unit": "lookups/s", "cores": n, "kind": "oracle", "sample": sample,
            "single_thread_value": one, "host": desc}


def copy_bandwidth(dev, mib=4096, reps=5):
    """Device-to-device copy of `mib` MiB (read + write bytes per second), the best of `reps`."""
    import torch

    n = (mib << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = float("inf")
    for _ in range(reps):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        dst.copy_(src)
        b.record()
        torch.cuda.synchronize()
        best = min(best, a.elapsed_time(b))
    del src, dst
    torch.cuda.empty_cache()
    return 2 * (mib << 20) / (best * 1e-3) / 1e9


def calibration_kernels(dev):
    """Kernels of known HBM traffic for the read-request and WRITE_SIZE counters: a 2 GiB copy,
    a 2 GiB streaming read (sum), and gathers of 1 GiB of random 512-byte rows and of
    random 64-byte rows out of 8 GiB tables (far beyond the 256 MB last-level cache)."""
    import torch

    g = torch.Generator(device=dev)
    g.manual_seed(7)
    n = (2 << 30) // 4
    a = torch.ones(n, dtype=torch.float32, device=dev)
    b = torch.empty_like(a)
    b.copy_(a)                                   # 2 GiB read, 2 GiB written
    s = a.sum()                                  # 2 GiB read
    del b
    big = torch.ones((8 << 30) // 4, dtype=torch.float32, device=dev)
    rows512 = big.view(-1, 128)
    i512 = torch.randint(0, rows512.shape[0], ((1 << 30) // 512,), generator=g, device=dev)
    r1 = rows512.index_select(0, i512)           # 1 GiB of 512-byte rows read, 1 GiB written
    rows64 = big.view(-1, 16)
    i64 = torch.randint(0, rows64.shape[0], ((1 << 30) // 64,), generator=g, device=dev)
    r2 = rows64.index_select(0, i64)             # 1 GiB of 64-byte rows read, 1 GiB written
    torch.cuda.synchronize()
    print(f"[bench] calibration kernels done (sum {float(s):.0f}, {r1.numel() + r2.numel()} gathered)",
          file=sys.stderr, flush=True)
    del a, big, r1, r2
    torch.cuda.empty_cache()


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5, help="untimed steps from the fresh state (timed separately "
                                                            "as the cold-cache steps)")
    ap.add_argument("--config", default="industrial")
    ap.add_argument("--table", choices=("device", "host"), default="device",
                    help="where the low-precision table lives (host: pinned host memory over the host link)")
    ap.add_argument("--set", action="append", default=[], metavar="KEY=VALUE",
                    help="override a field of the named workload (e.g. bits=16); int, float or text")
    ap.add_argument("--pool", type=int, default=3, help="distinct input batches cycled through")
    ap.add_argument("--stats-steps", type=int, default=3)
    ap.add_argument("--cpu-steps", type=int, default=60)
    ap.add_argument("--cpu-budget", type=float, default=12.0, help="oracle seconds per thread")
    ap.add_argument("--cpu-threads", type=int, default=0, help="oracle threads (0: usable host cores, at most 16)")
    ap.add_argument("--cpu-rows", type=int, default=0, help="cut each table to this many rows for the oracle")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-copy-bw", action="store_true")
    ap.add_argument("--calibration", action="store_true",
                    help="first run kernels of known HBM traffic (for the HBM read and write counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the multi-GPU path is not built.",
              file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2010_11305_amd.emb_cache import EmbCache

    over = {}
    for kv in args.set:
        k, v = kv.split("=", 1)
        for conv in (int, float):
            try:
                v = conv(v)
                break
            except ValueError:
                pass
        over[k] = v
    cfg = configs.get(args.config, **over)
    T, B, d = len(cfg["rows"]), cfg["batch"], cfg["dim"]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.calibration:
        calibration_kernels(dev)
    copy_gbs = None if args.no_copy_bw else copy_bandwidth(dev)
    if copy_gbs is not None:
        print(f"[bench] device copy: {copy_gbs:.0f} GB/s (read + write)", file=sys.stderr, flush=True)

    t0 = time.time()
    pool = []
    for k in range(args.pool):
        idx, off = workload.make_indices(cfg, k)
        pool.append((torch.from_numpy(idx).to(dev), torch.from_numpy(off).to(dev), idx.size))
        print(f"[bench] input batch {k}: {idx.size} lookups ({time.time() - t0:.1f} s)", file=sys.stderr, flush=True)
    gen = torch.Generator(device=dev)
    gen.manual_seed(cfg["grad_seed"])
    grads = [torch.randn((B, T, d), generator=gen, device=dev, dtype=torch.float32) * cfg["grad_sigma"]
             for _ in range(2)]
    max_idx = max(p[2] for p in pool)
    emb = EmbCache(cfg, max_indices=max_idx, table=args.table)
    emb.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    out = torch.empty((B, T, d), dtype=torch.float32, device=dev)
    torch.cuda.synchronize()
    print(f"[bench] state {emb.sizes.state_bytes / 2**30:.2f} GiB, workspace {emb.sizes.workspace_bytes / 2**30:.2f} GiB",
          file=sys.stderr, flush=True)

    def step(k, ev=None):
        idx, off, _ = pool[k % len(pool)]
        if ev is not None:
            ev[0].record()
        emb.forward(idx, off, B, out=out)
        if ev is not None:
            ev[1].record()
        emb.backward_update(idx, off, B, grads[k % 2])
        if ev is not None:
            ev[2].record()

    def events(n):
        return [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(n)]

    # the first steps after initialisation start from an empty cache: timed one by one
    cold = events(args.warmup)
    for k in range(args.warmup):
        step(k, cold[k])
    torch.cuda.synchronize()
    cold_ms = [e[0].elapsed_time(e[2]) for e in cold]
    print(f"[bench] warmup done ({args.warmup} steps from a fresh state)", file=sys.stderr, flush=True)

    emb.set_update_timing(True)  # HIP events around k_update, on the library's stream
    evs = events(args.steps)
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_start.record()
    for k in range(args.steps):
        step(args.warmup + k, evs[k])
    t_end.record()
    torch.cuda.synchronize()
    total_ms = t_start.elapsed_time(t_end)
    upd_ms = emb.update_times(args.steps)
    emb.set_update_timing(False)
    fwd_ms = [e[0].elapsed_time(e[1]) for e in evs]
    bwd_ms = [e[1].elapsed_time(e[2]) for e in evs]
    step_ms = [e[0].elapsed_time(e[2]) for e in evs]
    ms_per_step = total_ms / args.steps
    lookups = sum(pool[(args.warmup + k) % len(pool)][2] for k in range(args.steps))
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.3f} ms/step", file=sys.stderr, flush=True)

    # algorithmic bytes from the statistics of further steps of the same stream
    fwd_b, bwd_b, upd_b, grad_b, n_st = 0, 0, 0, 0, 0
    hit_lk, all_lk = 0, 0
    counts = {}
    for k in range(args.stats_steps):
        step(args.warmup + args.steps + k)
        for t in range(T):
            st = emb.stats(t)
            f, b = algorithmic_bytes(cfg, st, B)
            fwd_b += f
            bwd_b += b
            upd_b += update_kernel_bytes(cfg, st)
            grad_b += merged_gradient_bytes(cfg, st)
            hit_lk += st["hit_lookups"]
            all_lk += st["lookups"]
            for key in ("unique", "unique_hits", "inserts", "bypasses", "evictions", "hit_evictions"):
                counts[key] = counts.get(key, 0) + st[key]
        n_st += 1
    fwd_b /= n_st
    bwd_b /= n_st
    upd_b /= n_st
    grad_b /= n_st
    upd_avg = float(np.mean(upd_ms)) if len(upd_ms) else float("nan")
    upd_gbs = upd_b / (upd_avg * 1e-3) / 1e9
    status = emb.check()
    step_bytes = fwd_b + bwd_b
    gbs = step_bytes / (ms_per_step * 1e-3) / 1e9
    fwd_avg = float(np.mean(fwd_ms))
    fwd_gbs = fwd_b / (fwd_avg * 1e-3) / 1e9

    result = {
        "metric": METRIC,
        "value": lookups / (total_ms * 1e-3),
        "unit": "lookups/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": describe(cfg), "global_batch": B, "tables": T, "lookups_per_step": lookups / args.steps,
                   "table_memory": args.table},
        "hbm_gbps_algorithmic": gbs,
        "hbm_frac_of_peak": gbs / HBM_PEAK_GBS,
        "hbm_frac_of_copy": gbs / copy_gbs if copy_gbs else None,
        "bytes_per_step_algorithmic": step_bytes,
        "roofline_step": {"bound": "hbm", "what": "whole step (forward + backward_update), algorithmic bytes",
                          "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": gbs / HBM_PEAK_GBS,
                          "achievable": copy_gbs, "frac_of_achievable": gbs / copy_gbs if copy_gbs else None},
        "hbm_copy_gbps": copy_gbs,
        "ms_per_step_median": float(np.median(step_ms)),
        "ms_per_step_p90": float(np.percentile(step_ms, 90)),
        "cold_steps_ms": cold_ms,
        "fwd_ms": fwd_avg,
        "bwd_ms": float(np.mean(bwd_ms)),
        "fwd_ms_p90": float(np.percentile(fwd_ms, 90)),
        "bwd_ms_p90": float(np.percentile(bwd_ms, 90)),
        "hit_rate_lookups": hit_lk / max(all_lk, 1),
        "rows_per_step": {k: v / max(n_st, 1) for k, v in counts.items()},
        "status": status,
        "roofline": {"bound": "hbm", "kernel": "k_update (merged gradient, fetch, optimizer, write-back)",
                     "achieved": upd_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": upd_gbs / HBM_PEAK_GBS,
                     "traffic": measured_update_traffic(), "kernel_ms": upd_avg,
                     "algorithmic_bytes_per_launch": upd_b, "implementation_bytes_per_launch": grad_b},
        "roofline_forward": {"bound": "hbm", "kernels": "k_fwd_probe + k_fwd_gather (whole forward call)",
                             "achieved": fwd_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": fwd_gbs / HBM_PEAK_GBS, "algorithmic_bytes_per_call": fwd_b},
    }
    if not args.no_cpu_baseline:
        del emb, grads, pool, out
        torch.cuda.empty_cache()
        threads = args.cpu_threads or min(16, host_description()["nproc"] or 1)
        print(f"[bench] CPU oracle baseline, {threads} threads ...", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(cfg, args.cpu_steps, args.cpu_budget, threads, args.cpu_rows)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
