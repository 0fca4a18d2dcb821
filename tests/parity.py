"""Helpers of the GPU parity tests: one oracle and one GPU handle fed the same
seeded inputs; every piece of state compared after every step.

Bar: bit-exact for codes, scales, biases, tags, LRU stamps, LFU counts and
statistics; FP32 pooled outputs, cache rows and Adagrad state within a relative
error of 1e-5 (|a-b| <= 1e-5*|b| + 1e-30), and in practice bit-exact, which is
asserted too because every float operation of both sides is the same IEEE op.
"""
import sys

import numpy as np

from common import oracle_from_cfg
from paper_2010_11305_amd import workload

RTOL = 1e-5


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def assert_f32(a, b, what):
    a = np.asarray(a, dtype=np.float32)
    b = np.asarray(b, dtype=np.float32)
    assert a.shape == b.shape, what
    close = np.abs(a.astype(np.float64) - b.astype(np.float64)) <= RTOL * np.abs(b.astype(np.float64)) + 1e-30
    bad = np.nonzero(~close.ravel())[0]
    assert bad.size == 0, f"{what}: {bad.size} elements beyond 1e-5, first at {bad[:5]}"
    neq = np.nonzero(a.view(np.uint32).ravel() != b.view(np.uint32).ravel())[0]
    assert neq.size == 0, f"{what}: {neq.size} elements not bit-identical, first at {neq[:5]}"


def assert_same(a, b, what):
    a, b = np.asarray(a), np.asarray(b)
    neq = np.nonzero(a.ravel() != b.ravel())[0]
    assert neq.size == 0, f"{what}: {neq.size} mismatches, first at {neq[:5]}: {a.ravel()[neq[:5]]} vs {b.ravel()[neq[:5]]}"


def compare_state(o, g, cfg, tables=None, rows=None):
    tables = range(len(cfg["rows"])) if tables is None else tables
    for t in tables:
        n = cfg["rows"][t] if rows is None else min(rows, cfg["rows"][t])
        a, b = g.export_rows(t, 0, n), o.export_rows(t, 0, n)
        assert_same(a["codes"], b["codes"], f"codes t{t}")
        assert_same(a["scale"].view(np.uint32), b["scale"].view(np.uint32), f"scale t{t}")
        assert_same(a["bias"].view(np.uint32), b["bias"].view(np.uint32), f"bias t{t}")
        if cfg["policy"] == "lfu":
            assert_same(a["cnt"], b["cnt"], f"lfu counts t{t}")
        if cfg["optimizer"] == "adagrad":
            assert_f32(a["G"], b["G"], f"adagrad t{t}")
        if g.slots[t]:
            ca, cb = g.export_cache(t), o.export_cache(t)
            assert_same(ca["tag"], cb["tag"], f"tags t{t}")
            valid = cb["tag"] >= 0
            assert_f32(ca["crow"][valid], cb["crow"][valid], f"cache rows t{t}")
            if cfg["policy"] == "lru":
                assert_same(ca["ts"], cb["ts"], f"lru stamps t{t}")


def to_dev(st, torch):
    return (torch.from_numpy(st["indices"]).cuda(), torch.from_numpy(st["offsets"]).cuda(),
            torch.from_numpy(st["grad"]).cuda())


def make_pair(cfg, max_indices=None, table="device"):
    from paper_2010_11305_amd.emb_cache import EmbCache
    o = oracle_from_cfg(cfg)
    o.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    if max_indices is None:
        max_indices = max(1, int(workload.make_indices(cfg, 0)[0].size * 2 + 64))
    g = EmbCache(cfg, max_indices=max_indices, table=table)
    g.init_uniform(cfg["init_lo"], cfg["init_hi"], cfg["init_seed"])
    return o, g


def step_both(o, g, cfg, st, torch, check_out=True):
    idx, off, grad = to_dev(st, torch)
    B = st["batch"]
    out_g = g.forward(idx, off, B)
    out_o = o.forward(st["indices"], st["offsets"], B)
    if check_out:
        assert_f32(out_g.cpu().numpy(), out_o, "pooled output")
    g.backward_update(idx, off, B, grad)
    o.backward_update(st["indices"], st["offsets"], B, st["grad"])
    torch.cuda.synchronize()
    for t in range(len(cfg["rows"])):
        sg, so = g.stats(t), o.stats(t)
        assert sg == so, f"stats t{t}: gpu {sg} oracle {so}"
