"""ctypes binding of libembcache (include/emb_cache.h).

Argument marshalling only: every step of the training path runs in the HIP
kernels of the library.  torch provides the device buffers (state, workspace,
outputs) and the stream.  Raises if the library has not been built; there is no
fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libembcache.so")

EMB_OK, EMB_EINVAL, EMB_ENOMEM, EMB_EINDEX, EMB_EHIP = 0, 1, 2, 3, 4
STAT_NAMES = (
    "lookups", "hit_lookups", "bwd_lookups", "unique", "unique_hits", "inserts",
    "bypasses", "evictions", "empty_fills", "hit_evictions", "invalid_fwd", "invalid_bwd",
)
NSTAT = len(STAT_NAMES)


class EmbCacheError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__(f"{what}: {status_string(status)} (status {status})")


class Config(ctypes.Structure):
    _fields_ = [
        ("num_tables", ctypes.c_int32),
        ("dim", ctypes.c_int32),
        ("rows", ctypes.POINTER(ctypes.c_int64)),
        ("precision", ctypes.c_int32),
        ("sb_dtype", ctypes.c_int32),
        ("cache_fraction", ctypes.c_double),
        ("assoc", ctypes.c_int32),
        ("policy", ctypes.c_int32),
        ("lfu_decay_interval", ctypes.c_int32),
        ("rounding", ctypes.c_int32),
        ("optimizer", ctypes.c_int32),
        ("lr", ctypes.c_float),
        ("eps", ctypes.c_float),
        ("seed", ctypes.c_uint64),
        ("max_batch", ctypes.c_int32),
        ("max_indices", ctypes.c_int64),
    ]


class Sizes(ctypes.Structure):
    _fields_ = [
        ("state_bytes", ctypes.c_size_t),
        ("workspace_bytes", ctypes.c_size_t),
        ("total_rows", ctypes.c_int64),
        ("total_slots", ctypes.c_int64),
        ("row_bytes", ctypes.c_int32),
        ("pad", ctypes.c_int32),
        ("table_bytes", ctypes.c_size_t),
    ]


_lib = None


def load():
    """Load libembcache.so (no build here: build with paper_2010_11305_amd.build)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2010_11305_amd.build`")
    L = ctypes.CDLL(LIB_PATH)
    c, P = ctypes, ctypes.c_void_p
    i32, i64, u64, f32 = c.c_int32, c.c_int64, c.c_uint64, c.c_float
    sig = {
        "emb_cache_query_sizes": [c.POINTER(Config), c.POINTER(Sizes)],
        "emb_cache_table_geometry": [c.POINTER(Config), i32, c.POINTER(i64), c.POINTER(i64)],
        "emb_cache_create": [c.POINTER(Config), P, c.c_size_t, P, c.c_size_t, P, c.POINTER(P)],
        "emb_cache_create_with_table": [c.POINTER(Config), P, c.c_size_t, P, c.c_size_t, P, c.c_size_t, P,
                                        c.POINTER(P)],
        "emb_cache_destroy": [P],
        "emb_cache_init_uniform": [P, f32, f32, u64, P],
        "emb_cache_forward": [P, P, i64, P, i32, P, P],
        "emb_cache_forward_noalloc": [P, P, i64, P, i32, P, P],
        "emb_cache_backward_update": [P, P, i64, P, i32, P, P],
        "emb_cache_get_stats": [P, i32, P, P],
        "emb_cache_check": [P, P],
        "emb_cache_export_rows": [P, i32, i64, i64, P, P, P, P, P, P],
        "emb_cache_import_rows": [P, i32, i64, i64, P, P, P, P, P, P],
        "emb_cache_export_cache": [P, i32, P, P, P, P],
        "emb_cache_import_cache": [P, i32, P, P, P, P],
        "emb_cache_get_step": [P, c.POINTER(u64)],
        "emb_cache_set_step": [P, u64],
        "emb_cache_set_update_timing": [P, i32],
        "emb_cache_get_update_times": [P, P, i32, c.POINTER(i32)],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = c.c_int
    L.emb_cache_status_string.argtypes = [c.c_int]
    L.emb_cache_status_string.restype = c.c_char_p
    _lib = L
    return L


def status_string(status: int) -> str:
    try:
        return load().emb_cache_status_string(int(status)).decode()
    except Exception:  # library missing while formatting an error
        return "status"


def _check(st: int, what: str):
    if st != EMB_OK:
        raise EmbCacheError(st, what)


def make_config(cfg: dict, max_indices: int, max_batch: int | None = None):
    """C config from a workload dict (see configs.py).  Returns (Config, keepalive)."""
    rows = (ctypes.c_int64 * len(cfg["rows"]))(*[int(r) for r in cfg["rows"]])
    c = Config()
    c.num_tables = len(cfg["rows"])
    c.dim = int(cfg["dim"])
    c.rows = rows
    c.precision = int(cfg["bits"])
    c.sb_dtype = 1 if cfg.get("sb_fp16") else 0
    c.cache_fraction = float(cfg["cache_fraction"])
    c.assoc = int(cfg["assoc"])
    c.policy = 0 if cfg["policy"] == "lru" else 1
    c.lfu_decay_interval = int(cfg.get("lfu_decay_interval", 0))
    c.rounding = 1 if cfg["rounding"] == "stochastic" else 0
    c.optimizer = 1 if cfg["optimizer"] == "adagrad" else 0
    c.lr = float(cfg["lr"])
    c.eps = float(cfg.get("eps", 1e-8))
    c.seed = int(cfg["seed"])
    c.max_batch = int(max_batch if max_batch is not None else cfg["batch"])
    c.max_indices = int(max_indices)
    return c, rows


def query_sizes(cfg: dict, max_indices: int, max_batch: int | None = None) -> dict:
    c, keep = make_config(cfg, max_indices, max_batch)
    s = Sizes()
    _check(load().emb_cache_query_sizes(ctypes.byref(c), ctypes.byref(s)), "emb_cache_query_sizes")
    del keep
    return {"state_bytes": s.state_bytes, "workspace_bytes": s.workspace_bytes, "total_rows": s.total_rows,
            "total_slots": s.total_slots, "row_bytes": s.row_bytes, "table_bytes": s.table_bytes}


def _np(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _dptr(t):
    return ctypes.c_void_p(t.data_ptr())


class EmbCache:
    """Handle over torch-allocated device buffers.

    forward(indices, offsets, batch) -> pooled [batch][T][dim] FP32 (torch, device)
    backward_update(indices, offsets, batch, grad_out)

    table="host" puts the low-precision table in pinned host memory (torch
    pin_memory, i.e. hipHostMalloc) that the kernels reach over the host link; the
    FP32 cache and everything else stay in device memory.
    """

    def __init__(self, cfg: dict, max_indices: int, max_batch: int | None = None, device=None, table="device"):
        import torch

        self.torch = torch
        self.cfg = dict(cfg)
        self.T = len(cfg["rows"])
        self.dim = int(cfg["dim"])
        # exported codes: binary16 bit patterns for an FP16 table, else one code per byte
        self.code_dtype = np.uint16 if int(cfg["bits"]) == 16 else np.uint8
        self.device = torch.device(device or "cuda")
        self._c, self._keep = make_config(cfg, max_indices, max_batch)
        L = load()
        s = Sizes()
        _check(L.emb_cache_query_sizes(ctypes.byref(self._c), ctypes.byref(s)), "emb_cache_query_sizes")
        self.sizes = s
        self.workspace = torch.empty(max(int(s.workspace_bytes), 256), dtype=torch.uint8, device=self.device)
        h = ctypes.c_void_p()
        if table == "device":
            self.state = torch.empty(max(int(s.state_bytes), 256), dtype=torch.uint8, device=self.device)
            self.table = None
            _check(L.emb_cache_create(ctypes.byref(self._c), _dptr(self.state), s.state_bytes,
                                      _dptr(self.workspace), s.workspace_bytes, self._stream(), ctypes.byref(h)),
                   "emb_cache_create")
        elif table == "host":
            core = int(s.state_bytes - s.table_bytes)
            self.state = torch.empty(max(core, 256), dtype=torch.uint8, device=self.device)
            # 256 bytes of slack so that the table can start on a 256-byte boundary
            self._table_mem = torch.empty(int(s.table_bytes) + 256, dtype=torch.uint8, pin_memory=True)
            skip = (-self._table_mem.data_ptr()) % 256
            self.table = self._table_mem[skip:skip + int(s.table_bytes)]
            _check(L.emb_cache_create_with_table(ctypes.byref(self._c), _dptr(self.state), core,
                                                 ctypes.c_void_p(self.table.data_ptr()), s.table_bytes,
                                                 _dptr(self.workspace), s.workspace_bytes, self._stream(),
                                                 ctypes.byref(h)), "emb_cache_create_with_table")
        else:
            raise ValueError(f"table must be 'device' or 'host', not {table!r}")
        self._h = h
        self.n_sets, self.slots = [], []
        for t in range(self.T):
            ns, sl = ctypes.c_int64(), ctypes.c_int64()
            _check(L.emb_cache_table_geometry(ctypes.byref(self._c), t, ctypes.byref(ns), ctypes.byref(sl)),
                   "emb_cache_table_geometry")
            self.n_sets.append(ns.value)
            self.slots.append(sl.value)

    def _stream(self):
        return ctypes.c_void_p(self.torch.cuda.current_stream(self.device).cuda_stream)

    def close(self):
        if getattr(self, "_h", None):
            load().emb_cache_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # ---- training step ------------------------------------------------------------------
    def init_uniform(self, lo=-0.05, hi=0.05, init_seed=1):
        _check(load().emb_cache_init_uniform(self._h, lo, hi, int(init_seed), self._stream()), "init_uniform")

    def _inputs(self, indices, offsets, batch):
        torch = self.torch
        assert indices.dtype == torch.int32 and offsets.dtype == torch.int32
        assert indices.is_cuda and offsets.is_cuda and indices.is_contiguous() and offsets.is_contiguous()
        assert offsets.numel() == self.T * batch + 1
        return _dptr(indices), indices.numel(), _dptr(offsets)

    def forward(self, indices, offsets, batch, out=None):
        torch = self.torch
        ip, n, op = self._inputs(indices, offsets, batch)
        if out is None:
            out = torch.empty((batch, self.T, self.dim), dtype=torch.float32, device=self.device)
        assert out.shape == (batch, self.T, self.dim) and out.is_contiguous() and out.dtype == torch.float32
        _check(load().emb_cache_forward(self._h, ip, n, op, int(batch), _dptr(out), self._stream()), "forward")
        return out

    def forward_noalloc(self, indices, offsets, batch, out):
        """emb_cache_forward_noalloc: the forward with the library's static scratch in place
        of the workspace; `out` is the caller's (nothing is allocated here either)."""
        torch = self.torch
        ip, n, op = self._inputs(indices, offsets, batch)
        assert out.shape == (batch, self.T, self.dim) and out.is_contiguous() and out.dtype == torch.float32
        _check(load().emb_cache_forward_noalloc(self._h, ip, n, op, int(batch), _dptr(out), self._stream()),
               "forward_noalloc")
        return out

    def backward_update(self, indices, offsets, batch, grad_out):
        torch = self.torch
        ip, n, op = self._inputs(indices, offsets, batch)
        assert grad_out.shape == (batch, self.T, self.dim) and grad_out.dtype == torch.float32
        assert grad_out.is_cuda and grad_out.is_contiguous()
        _check(load().emb_cache_backward_update(self._h, ip, n, op, int(batch), _dptr(grad_out), self._stream()),
               "backward_update")

    # ---- inspection -----------------------------------------------------------------------
    def stats(self, t: int) -> dict:
        out = np.zeros(NSTAT, dtype=np.int64)
        _check(load().emb_cache_get_stats(self._h, t, _np(out), self._stream()), "get_stats")
        return dict(zip(STAT_NAMES, (int(v) for v in out)))

    def check(self) -> int:
        return int(load().emb_cache_check(self._h, self._stream()))

    @property
    def step(self) -> int:
        v = ctypes.c_uint64()
        _check(load().emb_cache_get_step(self._h, ctypes.byref(v)), "get_step")
        return int(v.value)

    @step.setter
    def step(self, s: int):
        _check(load().emb_cache_set_step(self._h, int(s)), "set_step")

    # ---- measurement ----------------------------------------------------------------------
    def set_update_timing(self, enable: bool):
        _check(load().emb_cache_set_update_timing(self._h, 1 if enable else 0), "set_update_timing")

    def update_times(self, max_n: int = 64) -> np.ndarray:
        """Durations (ms) of the row-update kernel in the last timed backward calls."""
        ms = np.zeros(max_n, dtype=np.float32)
        n = ctypes.c_int32()
        _check(load().emb_cache_get_update_times(self._h, _np(ms), max_n, ctypes.byref(n)), "get_update_times")
        return ms[: n.value].copy()

    def export_rows(self, t: int, row0: int = 0, n: int | None = None) -> dict:
        n = int(self.cfg["rows"][t]) - row0 if n is None else n
        codes = np.empty((n, self.dim), dtype=self.code_dtype)
        scale = np.empty(n, dtype=np.float32)
        bias = np.empty(n, dtype=np.float32)
        cnt = np.empty(n, dtype=np.int32)
        G = np.empty(n, dtype=np.float32)
        _check(load().emb_cache_export_rows(self._h, t, row0, n, _np(codes), _np(scale), _np(bias), _np(cnt), _np(G),
                                            self._stream()), "export_rows")
        return {"codes": codes, "scale": scale, "bias": bias, "cnt": cnt, "G": G}

    def import_rows(self, t: int, row0: int, codes, scale, bias, cnt=None, G=None):
        arrs = [np.ascontiguousarray(a, dtype=dt) if a is not None else None
                for a, dt in zip([codes, scale, bias, cnt, G],
                                 [self.code_dtype, np.float32, np.float32, np.int32, np.float32])]
        n = len(next(a for a in arrs if a is not None))
        _check(load().emb_cache_import_rows(self._h, t, row0, n, *[_np(a) for a in arrs], self._stream()),
               "import_rows")

    def export_cache(self, t: int) -> dict:
        sl = self.slots[t]
        crow = np.empty((sl, self.dim), dtype=np.float32)
        tag = np.empty(sl, dtype=np.int32)
        ts = np.empty(sl, dtype=np.int32)
        _check(load().emb_cache_export_cache(self._h, t, _np(crow), _np(tag), _np(ts), self._stream()), "export_cache")
        return {"crow": crow, "tag": tag, "ts": ts}

    def import_cache(self, t: int, crow=None, tag=None, ts=None):
        arrs = [np.ascontiguousarray(a, dtype=dt) if a is not None else None
                for a, dt in zip([crow, tag, ts], [np.float32, np.int32, np.int32])]
        _check(load().emb_cache_import_cache(self._h, t, *[_np(a) for a in arrs], self._stream()), "import_cache")
