"""Hit-rate study on synthetic index streams (policy, associativity, cache size).

The paper reports cache hit rates for the Criteo-Kaggle tables (Sec. 4.3: direct-
mapped LRU < direct-mapped LFU < 32-way LFU at every size, on a stationary access
pattern) and for its internal data (Sec. 5.2: LRU ahead of LFU for small caches on the
largest tables, explained by a "data shift": ids popular for a while that later fade).
Neither data set is here.  This driver runs the GPU library on two synthetic streams
of the same kinds and reports the forward hit rate per lookup (hits / lookups):

* stationary: one table of 1M rows, one lookup per sample, Zipf(1.05) popularity;
* drift: the same, with the hot rows moved to other ids every 10 steps.

It reproduces the shape of those tables (which policy wins where), not their values.

    python -m paper_2010_11305_amd.hitrate [--steps 200] [--json out.json]
"""
from __future__ import annotations

import argparse
import json
import sys

import numpy as np

from . import configs, workload

STREAMS = {
    "stationary": dict(rows=[1_000_000], dim=16, bits=8, batch=16384, pooling=("fixed", 1), zipf=1.05),
    "drift": dict(rows=[1_000_000], dim=16, bits=8, batch=16384, pooling=("fixed", 1), zipf=1.05,
                  drift=(10, 0.37)),
}

# (stream, cache fraction, label, associativity, policy, LFU decay interval)
GRID = (
    [("stationary", f, lab, a, p, 0) for f in (0.05, 0.10, 0.30, 0.50)
     for lab, a, p in (("LRU", 1, "lru"), ("LFU", 1, "lfu"), ("32-way LFU", 32, "lfu"))]
    + [(s, f, lab, 32, p, dec) for s in ("stationary", "drift") for f in (0.001, 0.01, 0.10)
       for lab, p, dec in (("32-way LRU", "lru", 0), ("32-way LFU", "lfu", 0), ("32-way LFU, halved /10", "lfu", 10))]
)


def stream(name: str, steps: int):
    cfg = configs.get("tiny", **STREAMS[name])
    return cfg, [workload.make_indices(cfg, k) for k in range(steps)]


def hit_rate(cfg: dict, steps_idx, warm: int) -> float:
    """Forward hits / lookups over the steps after `warm`, on the GPU library."""
    import torch
    from .emb_cache import EmbCache

    dev = torch.device("cuda:0")
    L = max(i.size for i, _ in steps_idx)
    emb = EmbCache(cfg, max_indices=L)
    emb.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    B, T, d = cfg["batch"], len(cfg["rows"]), cfg["dim"]
    grad = torch.zeros((B, T, d), dtype=torch.float32, device=dev)
    out = torch.empty((B, T, d), dtype=torch.float32, device=dev)
    hits = looks = 0
    for k, (idx, off) in enumerate(steps_idx):
        it, ot = torch.from_numpy(idx).to(dev), torch.from_numpy(off).to(dev)
        emb.forward(it, ot, B, out=out)
        if k >= warm:
            s = emb.stats(0)
            hits += s["hit_lookups"]
            looks += s["lookups"]
        emb.backward_update(it, ot, B, grad)
    emb.close()
    return hits / max(looks, 1)


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--json", default=None)
    args = ap.parse_args(argv)
    warm = args.steps // 2
    data = {name: stream(name, args.steps) for name in STREAMS}
    rows = []
    for sname, frac, label, assoc, policy, decay in GRID:
        base, idx = data[sname]
        cfg = dict(base, cache_fraction=frac, assoc=assoc, policy=policy, lfu_decay_interval=decay)
        h = hit_rate(cfg, idx, warm)
        rows.append({"stream": sname, "cache_fraction": frac, "policy": label, "hit_rate": h})
        print(f"{sname:10s} {frac:6.1%} {label:24s} {h:7.2%}", flush=True)
    if args.json:
        with open(args.json, "w") as f:
            json.dump({"steps": args.steps, "warm": warm, "streams": {k: {kk: vv for kk, vv in v.items()}
                                                                   for k, v in STREAMS.items()},
                       "rows": rows}, f, indent=1)
    return 0


if __name__ == "__main__":
    sys.exit(main())
