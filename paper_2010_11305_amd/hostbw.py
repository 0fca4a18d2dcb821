"""Effective bandwidth against cache hit rate, with the low-precision table in device
memory or in pinned host memory (the experiment of Fig. 9 in Sec. 5.2, "Speed improvement").

The paper puts a large FP16 table in unified memory and the FP32 LRU cache in device
memory, and plots the effective bandwidth of the forward and backward passes against
the hit rate, between two bounds: the table in device memory and the table in
unified memory without a cache.  Here the table is either in device memory or in
pinned host memory that the kernels reach over the host link (emb_cache_create_with_table);
the cache size sets the hit rate.

Effective bandwidth = FP32 bytes of the rows a pass serves / pass time:
  forward:  lookups x 4d (one FP32 row per lookup, pooled);
  backward: unique rows x 2 x 4d (each updated row read and written once).

    python -m paper_2010_11305_amd.hostbw [--tables 10] [--steps 6] [--json out.json]
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np

from . import configs, workload

FRACTIONS = (0.0, 0.001, 0.002, 0.005, 0.01, 0.02, 0.05)


def measure(cfg: dict, table: str, pool, steps: int, warm: int = 2) -> dict:
    import torch
    from .emb_cache import EmbCache

    dev = torch.device("cuda:0")
    B, T, d = cfg["batch"], len(cfg["rows"]), cfg["dim"]
    L = max(i.numel() for i, _ in pool)
    emb = EmbCache(cfg, max_indices=L, table=table)
    emb.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    grad = torch.randn((B, T, d), device=dev) * 0.01
    out = torch.empty((B, T, d), device=dev)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    fwd, bwd, looks, hits, uniq = [], [], 0, 0, 0
    for k in range(warm + steps):
        it, ot = pool[k % len(pool)]
        ev[0].record()
        emb.forward(it, ot, B, out=out)
        ev[1].record()
        torch.cuda.synchronize()
        if k >= warm:
            st = [emb.stats(t) for t in range(T)]
            looks += sum(s["lookups"] for s in st)
            hits += sum(s["hit_lookups"] for s in st)
        emb.backward_update(it, ot, B, grad)
        ev[2].record()
        torch.cuda.synchronize()
        if k >= warm:
            uniq += sum(emb.stats(t)["unique"] for t in range(T))
            fwd.append(ev[0].elapsed_time(ev[1]))
            bwd.append(ev[1].elapsed_time(ev[2]))
    emb.close()
    f_ms, b_ms = float(np.median(fwd)), float(np.median(bwd))
    return {
        "table": table, "cache_fraction": cfg["cache_fraction"], "hit_rate": hits / max(looks, 1),
        "fwd_ms": f_ms, "bwd_ms": b_ms,
        "fwd_gbps": looks / steps * 4 * d / (f_ms * 1e-3) / 1e9,
        "bwd_gbps": uniq / steps * 8 * d / (b_ms * 1e-3) / 1e9,
        "lookups_per_s": looks / steps / ((f_ms + b_ms) * 1e-3),
    }


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--tables", type=int, default=10)
    ap.add_argument("--steps", type=int, default=6)
    ap.add_argument("--bits", type=int, default=16)
    ap.add_argument("--json", default=None)
    args = ap.parse_args(argv)
    import torch

    base = configs.get("industrial", rows=[5_000_000] * args.tables, bits=args.bits)
    dev = torch.device("cuda:0")
    pool = []
    for k in range(3):
        idx, off = workload.make_indices(base, k)
        pool.append((torch.from_numpy(idx).to(dev), torch.from_numpy(off).to(dev)))
    rows = []
    for table in ("device", "host"):
        for frac in FRACTIONS:
            r = measure(dict(base, cache_fraction=frac), table, pool, args.steps)
            rows.append(r)
            print(f"{table:6s} cache {frac:6.1%} hit {r['hit_rate']:7.2%}  fwd {r['fwd_ms']:8.2f} ms "
                  f"{r['fwd_gbps']:7.1f} GB/s  bwd {r['bwd_ms']:8.2f} ms {r['bwd_gbps']:7.1f} GB/s  "
                  f"{r['lookups_per_s'] / 1e9:6.3f} G lookups/s", flush=True)
    if args.json:
        with open(args.json, "w") as f:
            json.dump({"workload": dict(base, rows=f"{args.tables} x 5000000"), "rows": rows}, f, indent=1,
                      default=str)
    return 0


if __name__ == "__main__":
    sys.exit(main())
