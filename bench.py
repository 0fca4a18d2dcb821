"""Throughput of the cached mixed-precision EmbeddingBag training step on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config industrial] [--gpus 1]

One step = forward (tag probe, gather + dequantize, sum-pool) + backward_update
(sort/de-dup, merged gradients, priority update, replacement, optimizer, write-back,
evict/fill) over one batch of synthetic Zipf-skewed lookups already resident in
HBM.  Prints one JSON line: pooled lookups/s (value), algorithmic HBM GB/s, the
roofline of the dominant kernel, and the CPU oracle timed on a bounded sample.
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
    """HBM bytes per k_update launch from the committed counter summary (FETCH_SIZE x 2 +
    WRITE_SIZE x 1, see that file's calibration), or None when the summary was taken on
    other kernel sources."""
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
    """Algorithmic bytes of the row-update kernel (k_update) for one table and one step.

    It handles every unique row except the residents displaced after their own update
    (E_h, handled with the evictions): per row it reads the row (phi from the cache
    for a hit, rho from T for a miss) and the merged gradient (phi), reads and writes the
    Adagrad accumulator (8), and writes the row to its slot (phi: hit or insert) or to
    T (rho: bypass), plus tag and LRU stamp of an insert (8; 4 under LFU).
    """
    d = cfg["dim"]
    phi = 4 * d
    rho = record_bytes(cfg)
    U, Uh, Eh = st["unique"], st["unique_hits"], st["hit_evictions"]
    Uins, Ubyp = st["inserts"], st["bypasses"]
    rows = U - Eh
    b = phi * (Uh - Eh) + rho * (Uins + Ubyp) + phi * rows
    b += phi * (Uh - Eh) + phi * Uins + rho * Ubyp + (8 if cfg["policy"] == "lru" else 4) * Uins
    if cfg["optimizer"] == "adagrad":
        b += 8 * rows
    return b


def cpu_baseline(cfg, steps, budget_s):
    """The CPU oracle on one table of the workload (table 0), single thread."""
    import oracle  # test infrastructure: only this leg of the benchmark loads it

    one = dict(cfg, rows=[cfg["rows"][0]])
    o = oracle.Oracle(one["rows"], one["dim"], one["bits"], one["sb_fp16"], one["cache_fraction"], one["assoc"],
                      one["policy"], one.get("lfu_decay_interval", 0), one["rounding"] == "stochastic",
                      one["optimizer"] == "adagrad", one["lr"], one["eps"], one["seed"])
    o.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    B = cfg["batch"]
    lookups, elapsed, done = 0, 0.0, 0
    for k in range(steps):
        idx, off = workload.make_indices(cfg, k, tables=[0])
        n0 = int(off[B])
        g = workload._rng(cfg["grad_seed"], k, 99).standard_normal((B, 1, cfg["dim"]), dtype=np.float32)
        g *= np.float32(cfg["grad_sigma"])
        t0 = time.perf_counter()
        o.forward(idx[:n0], off[:B + 1], B)
        o.backward_update(idx[:n0], off[:B + 1], B, g)
        elapsed += time.perf_counter() - t0
        lookups += n0
        done += 1
        if elapsed > budget_s:
            break
    return {"value": lookups / elapsed, "unit": "lookups/s", "cores": 1, "kind": "oracle",
            "sample": f"table 0 of {len(cfg['rows'])} ({cfg['rows'][0]} rows), {done} steps of fwd+bwd+update, "
                      f"{lookups} lookups in {elapsed:.1f} s, single thread"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="industrial")
    ap.add_argument("--table", choices=("device", "host"), default="device",
                    help="where the low-precision table lives (host: pinned host memory over the host link)")
    ap.add_argument("--set", action="append", default=[], metavar="KEY=VALUE",
                    help="override a field of the named workload (e.g. bits=16); int, float or text")
    ap.add_argument("--pool", type=int, default=3, help="distinct input batches cycled through")
    ap.add_argument("--stats-steps", type=int, default=3)
    ap.add_argument("--cpu-steps", type=int, default=60)
    ap.add_argument("--cpu-budget", type=float, default=15.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="run one device-to-device copy of this size first (HBM counter calibration)")
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
    if args.copy_calibration:
        n = args.copy_calibration << 20
        src = torch.ones(n // 4, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        print(f"[bench] calibration copy: {n} bytes read, {n} bytes written", file=sys.stderr, flush=True)
        del src, dst

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

    for k in range(args.warmup):
        step(k)
    torch.cuda.synchronize()
    print(f"[bench] warmup done ({args.warmup} steps)", file=sys.stderr, flush=True)

    emb.set_update_timing(True)  # HIP events around k_update, on the library's stream
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
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
    ms_per_step = total_ms / args.steps
    lookups = sum(pool[(args.warmup + k) % len(pool)][2] for k in range(args.steps))
    print(f"[bench] timed {args.steps} steps: {ms_per_step:.3f} ms/step", file=sys.stderr, flush=True)

    # algorithmic bytes from the statistics of further steps of the same stream
    fwd_b, bwd_b, upd_b, n_st = 0, 0, 0, 0
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
            hit_lk += st["hit_lookups"]
            all_lk += st["lookups"]
            for key in ("unique", "unique_hits", "inserts", "bypasses", "evictions", "hit_evictions"):
                counts[key] = counts.get(key, 0) + st[key]
        n_st += 1
    fwd_b /= n_st
    bwd_b /= n_st
    upd_b /= n_st
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
        "bytes_per_step_algorithmic": step_bytes,
        "fwd_ms": fwd_avg,
        "bwd_ms": float(np.mean(bwd_ms)),
        "fwd_ms_p90": float(np.percentile(fwd_ms, 90)),
        "bwd_ms_p90": float(np.percentile(bwd_ms, 90)),
        "hit_rate_lookups": hit_lk / max(all_lk, 1),
        "rows_per_step": {k: v / max(n_st, 1) for k, v in counts.items()},
        "status": status,
        "roofline": {"bound": "hbm", "kernel": "k_update (merged gradient, fetch, row-wise Adagrad, write-back)",
                     "achieved": upd_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": upd_gbs / HBM_PEAK_GBS,
                     "traffic": measured_update_traffic(), "kernel_ms": upd_avg,
                     "algorithmic_bytes_per_launch": upd_b},
        "roofline_forward": {"bound": "hbm", "kernels": "k_fwd_probe + k_fwd_gather (whole forward call)",
                             "achieved": fwd_gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": fwd_gbs / HBM_PEAK_GBS, "algorithmic_bytes_per_call": fwd_b},
    }
    if not args.no_cpu_baseline:
        print("[bench] CPU oracle baseline ...", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(cfg, args.cpu_steps, args.cpu_budget)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
