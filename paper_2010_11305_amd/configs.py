"""Named workloads: table shapes, precision, cache, policy, optimizer, batch shape.

Pure data.  Row counts of the 26 Criteo-Kaggle-shaped tables are the paper's
Table 1 ("DLRM benchmark model embedding sizes"); the other shapes are the
synthetic stand-ins for the paper's Sec. 4 (CPU, Criteo-Kaggle) and Sec. 5
(industrial GPU) workloads.  No dataset records are used anywhere.
"""
from __future__ import annotations

import copy

# Sec. 4.3, Table 1: embedding table sizes of the DLRM benchmark model (26 tables).
TABLE1_ROWS = [
    4, 4, 11, 16, 18, 24, 28, 105, 306, 584, 634, 1461, 2173, 3195, 5653, 5684,
    12518, 14993, 93146, 142572, 286181, 2202608, 5461306, 7046547, 8351593, 10131227,
]

_BASE = dict(
    sb_fp16=False, lfu_decay_interval=0, eps=1e-8, grad_sigma=0.01,
    init_lo=-0.05, init_hi=0.05, init_seed=1, seed=2, index_seed=3, grad_seed=4,
)

CONFIGS = {
    # 1 table x 1000 rows, d 16, INT8 + FP32 (s,b); 5% FP32 cache, 4-way LRU;
    # 128 bags of 1..4 lookups, Zipf 1.05; SGD lr 0.01; 10 steps.
    "tiny": dict(_BASE, rows=[1000], dim=16, bits=8, cache_fraction=0.05, assoc=4, policy="lru",
                 rounding="nearest", optimizer="sgd", lr=0.01, batch=128, pooling=("uniform", 1, 4),
                 zipf=1.05, steps=10),
    # 26 Table-1 tables, d 16, INT8 + FP32 (s,b); 5% cache 32-way LRU; batch 2048,
    # one lookup per table; Zipf 1.1; SGD lr 0.1; 100 steps.
    "kaggle_int8": dict(_BASE, rows=list(TABLE1_ROWS), dim=16, bits=8, cache_fraction=0.05, assoc=32,
                        policy="lru", rounding="nearest", optimizer="sgd", lr=0.1, batch=2048,
                        pooling=("fixed", 1), zipf=1.1, steps=100),
    # Same shapes in INT4 + FP16 (s,b); 1% cache 32-way LFU with counts halved every
    # 10 steps; stochastic rounding; row-wise Adagrad lr 0.01; batch 8192.
    "kaggle_int4": dict(_BASE, rows=list(TABLE1_ROWS), dim=16, bits=4, sb_fp16=True, cache_fraction=0.01,
                        assoc=32, policy="lfu", lfu_decay_interval=10, rounding="stochastic",
                        optimizer="adagrad", lr=0.01, batch=8192, pooling=("fixed", 1), zipf=1.1,
                        steps=100),
    # 100 tables x 5M rows x d 128, INT4 + FP16 (s,b) (34 GB of row records);
    # 1% cache 16-way LRU; 16384 bags per table, Poisson(30) lookups; Zipf 1.2;
    # row-wise Adagrad, stochastic rounding.
    "industrial": dict(_BASE, rows=[5_000_000] * 100, dim=128, bits=4, sb_fp16=True, cache_fraction=0.01,
                       assoc=16, policy="lru", rounding="stochastic", optimizer="adagrad", lr=0.01,
                       batch=16384, pooling=("poisson", 30), zipf=1.2, steps=25),
    # 1 table x 200M rows x d 256, INT8 + FP32 (s,b) (52.8 GB); 1% cache (2M rows)
    # 32-way LRU; 65536 bags of 64 lookups; Zipf 1.05; SGD lr 0.05; stochastic rounding.
    "stress": dict(_BASE, rows=[200_000_000], dim=256, bits=8, cache_fraction=0.01, assoc=32,
                   policy="lru", rounding="stochastic", optimizer="sgd", lr=0.05, batch=65536,
                   pooling=("fixed", 64), zipf=1.05, steps=25),
}

ORDER = ["tiny", "kaggle_int8", "kaggle_int4", "industrial", "stress"]


def get(name: str, **overrides) -> dict:
    cfg = copy.deepcopy(CONFIGS[name])
    cfg.update(overrides)
    cfg["name"] = name
    return cfg

