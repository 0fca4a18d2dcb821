"""Shared test helpers: build an oracle from a named config, tiny custom configs."""
import numpy as np

import oracle
from paper_2010_11305_amd import configs, workload


def oracle_from_cfg(cfg, **over):
    c = dict(cfg, **over)
    return oracle.Oracle(
        c["rows"], c["dim"], c["bits"], c["sb_fp16"], c["cache_fraction"], c["assoc"], c["policy"],
        c.get("lfu_decay_interval", 0), c["rounding"] == "stochastic", c["optimizer"] == "adagrad",
        c["lr"], c["eps"], c["seed"],
    )


def custom_cfg(**kw):
    """A small config derived from 'tiny' with overrides (rows, dim, bits, ...)."""
    return configs.get("tiny", **kw)


def effective_table(o, t):
    """FP32 view of table t: cache row when resident, else the dequantized row."""
    from exact import decode_rows
    r = o.export_rows(t)
    eff = decode_rows(r["codes"], r["scale"], r["bias"])
    c = o.export_cache(t)
    for k in np.nonzero(c["tag"] >= 0)[0]:
        eff[c["tag"][k]] = c["crow"][k]
    return eff


def exact_grad(cfg, step, scale_log2=-10, kmax=8):
    """Output gradients that are small multiples of 2^scale_log2, so that every
    sum of them up to a few thousand terms is exact in FP32 (order-free)."""
    T, B, d = len(cfg["rows"]), cfg["batch"], cfg["dim"]
    r = np.random.default_rng(1000 + step)
    k = r.integers(-kmax, kmax + 1, size=(B, T, d))
    return (k * 2.0**scale_log2).astype(np.float32)


__all__ = ["oracle_from_cfg", "custom_cfg", "effective_table", "exact_grad", "workload", "configs"]
