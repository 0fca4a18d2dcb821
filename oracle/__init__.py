"""CPU oracle for the cached mixed-precision EmbeddingBag step (test infrastructure).

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py``
may import this package.  It wraps ``emb_oracle.c`` (plain C, FP32, no fast-math)
through ctypes and shares nothing with the HIP library: not its header, not its
binding, not its state layout.  See the header comment of ``emb_oracle.c`` for
which part of the paper each function follows.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "emb_oracle.c")
_SO = os.path.join(_HERE, "liboracle.so")
_lib = None

NSTAT = 12
STAT_NAMES = (
    "lookups", "hit_lookups", "bwd_lookups", "unique", "unique_hits", "inserts",
    "bypasses", "evictions", "empty_fills", "hit_evictions", "invalid_fwd", "invalid_bwd",
)


def build() -> str:
    """Compile emb_oracle.c into liboracle.so (gcc, -O2, no FMA contraction)."""
    tmp = _SO + ".tmp"
    subprocess.check_call([
        "gcc", "-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
        _SRC, "-o", tmp, "-lm",
    ])
    os.replace(tmp, _SO)
    return _SO


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_SO):
            build()
        L = ctypes.CDLL(_SO)
        c = ctypes
        P = c.c_void_p
        L.orc_create.restype = P
        L.orc_create.argtypes = [c.POINTER(_Cfg), c.POINTER(c.c_int64)]
        L.orc_destroy.argtypes = [P]
        L.orc_geometry.restype = c.c_int64
        L.orc_geometry.argtypes = [P, c.c_int, c.POINTER(c.c_int64), c.POINTER(c.c_int64)]
        L.orc_get_step.restype = c.c_uint64
        L.orc_get_step.argtypes = [P]
        L.orc_set_step.argtypes = [P, c.c_uint64]
        L.orc_init_uniform.argtypes = [P, c.c_float, c.c_float, c.c_uint64]
        L.orc_forward.argtypes = [P, P, c.c_int64, P, c.c_int32, P]
        L.orc_backward_update.restype = c.c_int
        L.orc_backward_update.argtypes = [P, P, c.c_int64, P, c.c_int32, P]
        L.orc_stats.argtypes = [P, c.c_int, P]
        L.orc_export_rows.argtypes = [P, c.c_int, c.c_int64, c.c_int64, P, P, P, P, P]
        L.orc_import_rows.argtypes = [P, c.c_int, c.c_int64, c.c_int64, P, P, P, P, P]
        L.orc_export_cache.argtypes = [P, c.c_int, P, P, P]
        L.orc_import_cache.argtypes = [P, c.c_int, P, P, P]
        L.orc_philox4x32_10.argtypes = [P, P, P]
        L.orc_uniform.restype = c.c_float
        L.orc_uniform.argtypes = [c.c_uint64, c.c_uint32, c.c_uint32, c.c_uint32, c.c_uint32]
        L.orc_f32_to_f16_bits.restype = c.c_uint16
        L.orc_f32_to_f16_bits.argtypes = [c.c_float]
        L.orc_f16_bits_to_f32.restype = c.c_float
        L.orc_f16_bits_to_f32.argtypes = [c.c_uint16]
        L.orc_round_to_f16.restype = c.c_float
        L.orc_round_to_f16.argtypes = [c.c_float]
        L.orc_f16_round.restype = c.c_uint16
        L.orc_f16_round.argtypes = [c.c_float, c.c_int, c.c_float]
        L.orc_quantize_row.argtypes = [
            P, c.c_int, c.c_int, c.c_int, c.c_int, c.c_uint64, c.c_uint32, c.c_uint32, c.c_uint32,
            P, c.POINTER(c.c_float), c.POINTER(c.c_float),
        ]
        L.orc_compression_factor.restype = c.c_double
        L.orc_compression_factor.argtypes = [c.c_int, c.c_int, c.c_double, c.c_int, c.c_int]
        _lib = L
    return _lib


class _Cfg(ctypes.Structure):
    _fields_ = [
        ("num_tables", ctypes.c_int32),
        ("dim", ctypes.c_int32),
        ("bits", ctypes.c_int32),
        ("sb_fp16", ctypes.c_int32),
        ("cache_fraction", ctypes.c_double),
        ("assoc", ctypes.c_int32),
        ("policy", ctypes.c_int32),
        ("lfu_decay_interval", ctypes.c_int32),
        ("stochastic", ctypes.c_int32),
        ("adagrad", ctypes.c_int32),
        ("lr", ctypes.c_float),
        ("eps", ctypes.c_float),
        ("seed", ctypes.c_uint64),
    ]


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


class Oracle:
    """One oracle instance: tables, FP32 caches, policy state, step counter."""

    def __init__(self, rows, dim, bits, sb_fp16, cache_fraction, assoc, policy="lru",
                 lfu_decay_interval=0, stochastic=False, adagrad=False, lr=0.01, eps=1e-8, seed=2):
        self.rows = [int(r) for r in rows]
        self.T = len(self.rows)
        self.dim = int(dim)
        self.bits = int(bits)
        # an FP16 table exports its binary16 bit patterns; integer codes one per byte
        self.code_dtype = np.uint16 if self.bits == 16 else np.uint8
        self.sb_fp16 = bool(sb_fp16)
        self.policy = policy
        cfg = _Cfg(self.T, self.dim, self.bits, int(self.sb_fp16), float(cache_fraction), int(assoc),
                   0 if policy == "lru" else 1, int(lfu_decay_interval), int(bool(stochastic)),
                   int(bool(adagrad)), float(lr), float(eps), int(seed))
        rows_arr = (ctypes.c_int64 * self.T)(*self.rows)
        self._h = lib().orc_create(ctypes.byref(cfg), rows_arr)
        if not self._h:
            raise ValueError("oracle rejected the configuration")
        self.n_sets, self.slots = [], []
        for t in range(self.T):
            ns, sl = ctypes.c_int64(), ctypes.c_int64()
            lib().orc_geometry(self._h, t, ctypes.byref(ns), ctypes.byref(sl))
            self.n_sets.append(ns.value)
            self.slots.append(sl.value)

    def __del__(self):
        h = getattr(self, "_h", None)
        if h:
            lib().orc_destroy(h)
            self._h = None

    @property
    def step(self) -> int:
        return int(lib().orc_get_step(self._h))

    @step.setter
    def step(self, s: int) -> None:
        lib().orc_set_step(self._h, int(s))

    def init_uniform(self, lo=-0.05, hi=0.05, init_seed=1):
        lib().orc_init_uniform(self._h, lo, hi, int(init_seed))

    def forward(self, indices, offsets, batch):
        idx = np.ascontiguousarray(indices, dtype=np.int32)
        off = np.ascontiguousarray(offsets, dtype=np.int32)
        assert off.size == self.T * batch + 1
        out = np.empty((batch, self.T, self.dim), dtype=np.float32)
        lib().orc_forward(self._h, _ptr(idx), idx.size, _ptr(off), int(batch), _ptr(out))
        return out

    def backward_update(self, indices, offsets, batch, grad):
        idx = np.ascontiguousarray(indices, dtype=np.int32)
        off = np.ascontiguousarray(offsets, dtype=np.int32)
        g = np.ascontiguousarray(grad, dtype=np.float32)
        assert off.size == self.T * batch + 1 and g.shape == (batch, self.T, self.dim)
        # True when the call was rejected for malformed offsets (no state change; the step still counts)
        return bool(lib().orc_backward_update(self._h, _ptr(idx), idx.size, _ptr(off), int(batch), _ptr(g)))

    def stats(self, t):
        out = np.zeros(NSTAT, dtype=np.int64)
        lib().orc_stats(self._h, t, _ptr(out))
        return dict(zip(STAT_NAMES, (int(v) for v in out)))

    def export_rows(self, t, row0=0, n=None):
        n = self.rows[t] - row0 if n is None else n
        codes = np.empty((n, self.dim), dtype=self.code_dtype)
        scale = np.empty(n, dtype=np.float32)
        bias = np.empty(n, dtype=np.float32)
        cnt = np.empty(n, dtype=np.int32)
        G = np.empty(n, dtype=np.float32)
        lib().orc_export_rows(self._h, t, row0, n, _ptr(codes), _ptr(scale), _ptr(bias), _ptr(cnt), _ptr(G))
        return {"codes": codes, "scale": scale, "bias": bias, "cnt": cnt, "G": G}

    def import_rows(self, t, row0, codes=None, scale=None, bias=None, cnt=None, G=None):
        arrs = [codes, scale, bias, cnt, G]
        dts = [self.code_dtype, np.float32, np.float32, np.int32, np.float32]
        arrs = [None if a is None else np.ascontiguousarray(a, dtype=dt) for a, dt in zip(arrs, dts)]
        n = next(len(a) for a in arrs if a is not None)
        lib().orc_import_rows(self._h, t, row0, n, *[_ptr(a) for a in arrs])

    def export_cache(self, t):
        sl = self.slots[t]
        crow = np.empty((sl, self.dim), dtype=np.float32)
        tag = np.empty(sl, dtype=np.int32)
        ts = np.empty(sl, dtype=np.int32)
        lib().orc_export_cache(self._h, t, _ptr(crow), _ptr(tag), _ptr(ts))
        return {"crow": crow, "tag": tag, "ts": ts}

    def import_cache(self, t, crow=None, tag=None, ts=None):
        arrs = [None if a is None else np.ascontiguousarray(a, dtype=dt)
                for a, dt in zip([crow, tag, ts], [np.float32, np.int32, np.int32])]
        lib().orc_import_cache(self._h, t, *[_ptr(a) for a in arrs])


def philox4x32_10(counter, key):
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.empty(4, dtype=np.uint32)
    lib().orc_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


def uniform(seed, step, table, row, col) -> float:
    return float(lib().orc_uniform(seed, step, table, row, col))


def f32_to_f16_bits(x: float) -> int:
    return int(lib().orc_f32_to_f16_bits(x))


def f16_bits_to_f32(h: int) -> float:
    return float(lib().orc_f16_bits_to_f32(h))


def f16_round(x: float, stochastic: bool = False, u: float = 0.0) -> int:
    """Down-conversion of one value into binary16 bits: nearest-even, or stochastic
    with the uniform u (see orc_f16_round)."""
    return int(lib().orc_f16_round(x, int(bool(stochastic)), u))


def quantize_row(x, bits, sb_fp16=False, stochastic=False, seed=0, step=0, table=0, row=0):
    """Alg. 1 on one row: returns (codes uint8[d], scale, bias)."""
    xa = np.ascontiguousarray(x, dtype=np.float32)
    codes = np.empty(xa.size, dtype=np.uint8)
    s, b = ctypes.c_float(), ctypes.c_float()
    lib().orc_quantize_row(_ptr(xa), xa.size, bits, int(sb_fp16), int(stochastic), seed, step, table, row,
                           _ptr(codes), ctypes.byref(s), ctypes.byref(b))
    return codes, np.float32(s.value), np.float32(b.value)


def compression_factor(bits, D, ratio, counters=True, sb_bits=32) -> float:
    """Appendix memory compression factor (bits per row relative to FP32)."""
    return float(lib().orc_compression_factor(int(bits), int(D), float(ratio), int(bool(counters)), int(sb_bits)))
