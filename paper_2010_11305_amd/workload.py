"""Seeded synthetic inputs: index streams, bag offsets and output gradients.

This module holds none of the method's arithmetic; it only draws inputs.  Both
the CPU oracle and the HIP library are fed the arrays it returns.

* Indices of table t at step k: Zipf(alpha) ranks over [1, N_t] (the paper
  observes that under 20% of rows take over 80% of accesses), drawn by
  rejection-inversion (Hormann & Derflinger, 1996), then scattered over row ids
  by a seeded affine bijection row = (a*(rank-1) + c) mod N_t with gcd(a, N_t) = 1,
  so the hottest rows are not clustered in the low row ids or in one cache set.
* Popularity drift (optional, cfg["drift"] = (period, fraction)): the offset c of
  the bijection moves by fraction*N_t every `period` steps, so each popular row
  stays popular for a phase of `period` steps and then gives way to another one
  (the "data shift" of the paper's internal data, Sec. 5.2).
* Bag lengths: uniform U{lo..hi}, fixed, or Poisson(mean), per (table, bag).
* Offsets: int32 [T*B + 1], table-major (all bags of table 0, then table 1, ...).
* Output gradients: N(0, sigma) FP32 of shape [B][T][d].
Every draw comes from a numpy PCG64 stream keyed on (seed, step, table), so a
step's inputs do not depend on the order in which steps are generated.
"""
from __future__ import annotations

import math

import numpy as np


def _rng(*key) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([int(k) for k in key])))


class ZipfSampler:
    """Ranks k in [1, N] with P(k) proportional to k**-alpha (alpha > 0).

    Rejection-inversion: invert the integral H of the hat x**-alpha on the
    continuous range [1.5 - 1, N + 0.5], round, accept when the point falls under
    the histogram of the discrete pmf.  Vectorised; rejected draws are redrawn.
    """

    def __init__(self, N: int, alpha: float):
        if N < 1 or alpha <= 0:
            raise ValueError("need N >= 1 and alpha > 0")
        self.N = int(N)
        self.a = float(alpha)
        self.h_x1 = self._H(1.5) - 1.0
        self.h_n = self._H(self.N + 0.5)
        self.s = 2.0 - self._Hinv(self._H(2.5) - self._h(2.0))

    def _h(self, x):
        return np.exp(-self.a * np.log(x))

    def _H(self, x):
        # integral of t**-alpha from 1 to x: ((x**(1-alpha)) - 1) / (1 - alpha), log(x) at alpha = 1
        lx = np.log(x)
        t = (1.0 - self.a) * lx
        return np.where(np.abs(t) > 1e-8, np.expm1(t) / np.where(t == 0, 1, t), 1.0 + 0.5 * t) * lx

    def _Hinv(self, y):
        t = np.maximum(y * (1.0 - self.a), -1.0)
        f = np.where(np.abs(t) > 1e-8, np.log1p(t) / np.where(t == 0, 1, t), 1.0 - 0.5 * t)
        return np.exp(f * y)

    def sample(self, rng: np.random.Generator, n: int) -> np.ndarray:
        out = np.empty(n, dtype=np.int64)
        todo = np.arange(n)
        while todo.size:
            u = self.h_n + rng.random(todo.size) * (self.h_x1 - self.h_n)
            x = self._Hinv(u)
            k = np.clip(np.floor(x + 0.5), 1, self.N)
            ok = (k - x <= self.s) | (u >= self._H(k + 0.5) - self._h(k))
            out[todo[ok]] = k[ok].astype(np.int64)
            todo = todo[~ok]
        return out


def affine_bijection(seed: int, table: int, N: int):
    """(a, c) with gcd(a, N) = 1 so that rank -> (a*(rank-1) + c) mod N is a bijection."""
    if N <= 1:
        return 1, 0
    r = _rng(seed, table, 0xB17EC7)
    while True:
        a = int(r.integers(1, N))
        if math.gcd(a, N) == 1:
            break
    c = int(r.integers(0, N))
    return a, c


def bag_lengths(cfg: dict, step: int, table: int) -> np.ndarray:
    r = _rng(cfg["index_seed"], step, table, 1)
    kind = cfg["pooling"][0]
    B = cfg["batch"]
    if kind == "uniform":
        return r.integers(cfg["pooling"][1], cfg["pooling"][2] + 1, size=B).astype(np.int64)
    if kind == "fixed":
        return np.full(B, cfg["pooling"][1], dtype=np.int64)
    if kind == "poisson":
        return r.poisson(cfg["pooling"][1], size=B).astype(np.int64)
    raise ValueError(kind)


def table_indices(cfg: dict, step: int, table: int, n: int, sampler: ZipfSampler | None = None) -> np.ndarray:
    N = cfg["rows"][table]
    sampler = sampler or ZipfSampler(N, cfg["zipf"])
    ranks = sampler.sample(_rng(cfg["index_seed"], step, table, 2), n)
    a, c = affine_bijection(cfg["index_seed"], table, N)
    drift = cfg.get("drift")
    if drift:
        period, fraction = drift
        c = (c + (step // int(period)) * int(fraction * N)) % N
    return ((a * (ranks - 1) + c) % N).astype(np.int32)


def make_indices(cfg: dict, step: int, tables=None):
    """indices (int32 flat, table-major) and offsets (int32 [T*B+1]) for one step.

    `tables` restricts generation to a subset (the other tables get empty bags),
    which keeps single-table slices of large configs cheap.
    """
    T, B = len(cfg["rows"]), cfg["batch"]
    tables = range(T) if tables is None else tables
    lengths = np.zeros((T, B), dtype=np.int64)
    samplers = {}
    for t in tables:
        lengths[t] = bag_lengths(cfg, step, t)
    offsets = np.zeros(T * B + 1, dtype=np.int64)
    np.cumsum(lengths.ravel(), out=offsets[1:])
    if offsets[-1] >= 2**31:
        raise ValueError("more than 2^31 indices in one step")
    indices = np.empty(int(offsets[-1]), dtype=np.int32)
    for t in tables:
        key = (cfg["rows"][t], cfg["zipf"])
        if key not in samplers:
            samplers[key] = ZipfSampler(*key)
        p0, p1 = offsets[t * B], offsets[(t + 1) * B]
        indices[p0:p1] = table_indices(cfg, step, t, int(p1 - p0), samplers[key])
    return indices, offsets.astype(np.int32)


def make_grad(cfg: dict, step: int) -> np.ndarray:
    T, B, d = len(cfg["rows"]), cfg["batch"], cfg["dim"]
    r = _rng(cfg["grad_seed"], step)
    return (r.standard_normal((B, T, d), dtype=np.float32) * np.float32(cfg["grad_sigma"])).astype(np.float32)


def make_step(cfg: dict, step: int, tables=None):
    idx, off = make_indices(cfg, step, tables)
    return {"indices": idx, "offsets": off, "batch": cfg["batch"], "grad": make_grad(cfg, step)}
