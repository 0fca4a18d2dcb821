"""Pins of the oracle's cache replacement (Sec. 3 "Cache Replacement Policy", Alg. 2).

* One lookup per step into a single set of A ways: the cache must behave as
  textbook LRU (collections.OrderedDict) and as LFU with strictly-greater
  admission against the lowest-count resident (ties: lowest way).
* Direct-mapped LRU never compares priorities: every miss replaces the resident.
* Alg. 2 transcribed literally in Python, sequential over the step's sorted
  unique rows, on the paper's single-array emulation (one FP32 array, fake
  quantization of non-resident rows).  On streams where no set sees a hit after
  a miss in row order (and, for LFU, at most one unique row per set per step)
  the oracle's batched per-set rule must give the same tags and the same values.
"""
from collections import OrderedDict
from fractions import Fraction

import numpy as np
import pytest

import oracle
from common import custom_cfg, effective_table, oracle_from_cfg
from exact import dequant_exact, round_f32


def _one_lookup_step(o, r, g=None):
    idx = np.array([r], dtype=np.int32)
    off = np.array([0, 1], dtype=np.int32)
    if g is None:
        g = np.zeros((1, 1, o.dim), dtype=np.float32)
    o.backward_update(idx, off, 1, g)


@pytest.mark.parametrize("A", [2, 4, 8])
def test_single_set_lru_is_textbook_lru(A):
    N = 16 * A
    cfg = custom_cfg(rows=[N], cache_fraction=A / N, assoc=A, batch=1)
    o = oracle_from_cfg(cfg)
    o.init_uniform()
    assert o.n_sets == [1]
    lru = OrderedDict()
    rng = np.random.default_rng(A)
    for k in range(400):
        r = int(min(rng.zipf(1.3), N) - 1)
        if r in lru:
            lru.move_to_end(r)
        else:
            if len(lru) == A:
                lru.popitem(last=False)
            lru[r] = True
        _one_lookup_step(o, r)
        tags = o.export_cache(0)["tag"]
        assert set(int(t) for t in tags if t >= 0) == set(lru), k


@pytest.mark.parametrize("A,decay", [(4, 0), (8, 0), (4, 5)])
def test_single_set_lfu_strict_admission(A, decay):
    N = 16 * A
    cfg = custom_cfg(rows=[N], cache_fraction=A / N, assoc=A, batch=1, policy="lfu", lfu_decay_interval=decay)
    o = oracle_from_cfg(cfg)
    o.init_uniform()
    ways = [-1] * A
    cnt = np.zeros(N, dtype=np.int64)
    rng = np.random.default_rng(7 * A + decay)
    for k in range(400):
        if decay and k > 0 and k % decay == 0:
            cnt >>= 1
        r = int(min(rng.zipf(1.2), N) - 1)
        cnt[r] += 1
        if r not in ways:
            w = min(range(A), key=lambda w: (cnt[ways[w]], w) if ways[w] >= 0 else (-(2**62), w))
            if ways[w] < 0 or cnt[r] > cnt[ways[w]]:
                ways[w] = r
        _one_lookup_step(o, r)
        assert list(o.export_cache(0)["tag"]) == ways, k
        assert np.array_equal(o.export_rows(0)["cnt"], cnt)


def test_direct_mapped_lru_always_replaces():
    cfg = custom_cfg(rows=[64], cache_fraction=0.25, assoc=1, batch=6, pooling=("uniform", 1, 3))
    o = oracle_from_cfg(cfg)
    o.init_uniform()
    ns = o.n_sets[0]
    assert ns == 16
    from paper_2010_11305_amd import workload
    for k in range(30):
        st = workload.make_step(cfg, k)
        pre = o.export_cache(0)["tag"].copy()
        o.backward_update(st["indices"], st["offsets"], st["batch"], st["grad"])
        post = o.export_cache(0)["tag"]
        rows = set(int(r) for r in st["indices"])
        for s in range(ns):
            missed = [r for r in rows if r % ns == s and r != pre[s]]
            assert post[s] == (max(missed) if missed else pre[s])


# ---- literal Alg. 2 on the single-array emulation ----------------------------------------------
class LiteralAlg2:
    def __init__(self, o, cfg):
        self.cfg = cfg
        self.A = cfg["assoc"]
        self.ns = o.n_sets[0]
        self.N = cfg["rows"][0]
        self.W = effective_table(o, 0).copy()     # one FP32 array for table + cache
        self.IC = [[-1] * self.A for _ in range(self.ns)]
        self.PV = {}                               # per embedding row
        self.lr = Fraction(float(np.float32(cfg["lr"])))

    def pv(self, r):
        return -(2**62) if r < 0 else self.PV.get(r, 0)

    def fake_quantize(self, r, step):
        c, s, b = oracle.quantize_row(self.W[r], self.cfg["bits"], self.cfg["sb_fp16"],
                                      self.cfg["rounding"] == "stochastic", self.cfg["seed"], step, 0, r)
        self.W[r] = dequant_exact(c, s, b)

    def step(self, step, rows_counts, gsum):
        lru = self.cfg["policy"] == "lru"
        for i in sorted(rows_counts):                          # for i in I_U
            self.PV[i] = step if lru else self.PV.get(i, 0) + rows_counts[i]
            s = i % self.ns
            self.W[i] = np.array([round_f32(Fraction(float(self.W[i, j])) - self.lr * gsum[i][j])
                                  for j in range(self.W.shape[1])], dtype=np.float32)
            if i not in self.IC[s]:
                w = min(range(self.A), key=lambda w: (self.pv(self.IC[s][w]), w))
                j = self.IC[s][w]
                if not (self.A == 1 and lru) and self.PV[i] <= self.pv(j):
                    self.fake_quantize(i, step)                # bypass
                else:
                    if j >= 0:
                        self.fake_quantize(j, step)            # replace: evicted row to T
                    self.IC[s][w] = i


@pytest.mark.parametrize("policy,A,sr", [("lru", 4, False), ("lru", 2, True), ("lfu", 4, False),
                                         ("lfu", 2, True), ("lru", 1, False), ("lfu", 1, False)])
def test_batched_rule_matches_literal_alg2(policy, A, sr):
    N = 96
    cfg = custom_cfg(rows=[N], cache_fraction=(8 * A) / N, assoc=A, policy=policy, batch=6,
                     rounding="stochastic" if sr else "nearest", lr=0.5)
    o = oracle_from_cfg(cfg)
    o.init_uniform()
    lit = LiteralAlg2(o, cfg)
    ns = lit.ns
    rng = np.random.default_rng([len(policy), A, int(sr), 17])
    steps = 0
    tries = 0
    while steps < 40 and tries < 5000:
        tries += 1
        n = int(rng.integers(1, 7))
        idx = (np.minimum(rng.zipf(1.15, size=n), N) - 1).astype(np.int32)
        uniq = sorted(set(int(r) for r in idx))
        bysets = {}
        for r in uniq:
            bysets.setdefault(r % ns, []).append(r)
        ok = True
        for s, rs in bysets.items():
            if policy == "lfu" and len(rs) > 1:
                ok = False
            hits = [r for r in rs if r in lit.IC[s]]
            miss = [r for r in rs if r not in lit.IC[s]]
            if hits and miss and min(miss) < max(hits):
                ok = False
            if A == 1 and len(rs) > 1:
                ok = False
        if not ok:
            continue
        # one bag per lookup; gradients exact multiples of 2^-10 so sums are order-free
        B = len(idx)
        g = (rng.integers(-8, 9, size=(B, 1, 16)) * 2.0**-10).astype(np.float32)
        counts = {}
        gsum = {}
        for b, r in enumerate(idx):
            r = int(r)
            counts[r] = counts.get(r, 0) + 1
            acc = gsum.setdefault(r, [Fraction(0)] * 16)
            for j in range(16):
                acc[j] += Fraction(float(g[b, 0, j]))
        off = np.arange(B + 1, dtype=np.int32)
        lit.step(o.step, counts, gsum)
        o.backward_update(idx, off, B, g)
        tags = o.export_cache(0)["tag"].reshape(ns, A)
        assert [list(map(int, t)) for t in tags] == lit.IC, steps
        eff = effective_table(o, 0)
        assert np.array_equal(eff.view(np.uint32), lit.W.view(np.uint32)), steps
        steps += 1
    assert steps == 40
