"""Thin ctypes binding of libbgmf.so (the C ABI in include/bgmf.h).

Every function here only marshals arguments; all work runs in the HIP
library.  There is no fallback: if libbgmf.so is missing or cannot be
loaded, importing this module raises.
"""
from __future__ import annotations

import ctypes
import math
import os
import sys

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libbgmf.so")

BGMF_OK = 0
BGMF_E_ARG = -1
BGMF_E_STATE = -2
BGMF_E_RANGE = -3
BGMF_E_NONFINITE = -4
BGMF_E_NOMEM = -5
BGMF_E_BUDGET = -6
BGMF_E_HIP = -7
BGMF_E_UNSUPPORTED = -8
BGMF_E_TIMEOUT = -9

BGMF_OPT_SCHEDULE = 1
BGMF_OPT_WAIT_LIMIT_US = 2
BGMF_OPT_XCD_REMAP = 3
BGMF_OPT_RATINGS_BUDGET = 4
BGMF_OPT_STREAM_SLOTS = 5
BGMF_OPT_V_STAGING = 6
BGMF_OPT_PLACEMENT = 7
BGMF_OPT_STREAM_CHUNKS = 8
BGMF_OPT_RESIDENT_STRATA = 9
BGMF_OPT_BLOCK_PASSES = 10
BGMF_OPT_SINGLE_COLUMN = 11
BGMF_OPT_LDS_HANDOVER = 12
BGMF_OPT_TRACE = 13
BGMF_OPT_ALLOC_COUNT = 14
BGMF_OPT_LOAD_PEAK = 15
BGMF_OPT_LOAD_GROUPS = 16

EXPORTED = (
    "bgmf_create", "bgmf_destroy", "bgmf_last_error", "bgmf_set_stream", "bgmf_set_factors",
    "bgmf_load_coo", "bgmf_epoch", "bgmf_rmse", "bgmf_get_factors", "bgmf_get_layout",
    "bgmf_sync", "bgmf_factor_ptrs", "bgmf_set_option", "bgmf_get_option", "bgmf_get_timing",
    "bgmf_chain_stats", "bgmf_rmse_coo", "bgmf_fit", "bgmf_set_cuts", "bgmf_get_cuts",
    "bgmf_balanced_cuts", "bgmf_get_trace", "bgmf_query_sizes", "bgmf_bind",
    "bgmf_rmse_coo_dev", "bgmf_reorder_ids",
)


class BgmfError(RuntimeError):
    def __init__(self, code: int, message: str):
        super().__init__(f"[{code}] {message}")
        self.code = code


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is missing: build it with __graft_entry__.build() or "
                          "python -m paper_2304_13724_amd.build")
    lib = ctypes.CDLL(LIB_PATH)
    vp, I64, I32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32
    F32, c_int = ctypes.c_float, ctypes.c_int
    sig = {
        "bgmf_create": ([I64, I64, I32, I32], vp),
        "bgmf_destroy": ([vp], None),
        "bgmf_last_error": ([vp], ctypes.c_char_p),
        "bgmf_set_stream": ([vp, vp], c_int),
        "bgmf_set_factors": ([vp, vp, vp], c_int),
        "bgmf_load_coo": ([vp, vp, vp, vp, I64], c_int),
        "bgmf_epoch": ([vp, F32, F32], c_int),
        "bgmf_rmse": ([vp, ctypes.POINTER(ctypes.c_double)], c_int),
        "bgmf_get_factors": ([vp, vp, vp], c_int),
        "bgmf_get_layout": ([vp, vp, vp], c_int),
        "bgmf_sync": ([vp], c_int),
        "bgmf_factor_ptrs": ([vp, ctypes.POINTER(vp), ctypes.POINTER(vp)], c_int),
        "bgmf_set_option": ([vp, I32, I64], c_int),
        "bgmf_get_option": ([vp, I32, ctypes.POINTER(I64)], c_int),
        "bgmf_get_timing": ([vp, ctypes.POINTER(ctypes.c_double), ctypes.POINTER(ctypes.c_double)],
                            c_int),
        "bgmf_chain_stats": ([vp, vp], c_int),
        "bgmf_get_trace": ([vp, vp, vp, ctypes.POINTER(I64)], c_int),
        "bgmf_rmse_coo": ([vp, vp, vp, vp, I64, ctypes.POINTER(ctypes.c_double)], c_int),
        "bgmf_rmse_coo_dev": ([vp, vp, vp, vp, I64, ctypes.POINTER(ctypes.c_double)], c_int),
        "bgmf_fit": ([vp, F32, F32, I32, ctypes.c_double, ctypes.POINTER(I32), vp], c_int),
        "bgmf_set_cuts": ([vp, vp, vp], c_int),
        "bgmf_get_cuts": ([vp, vp, vp], c_int),
        "bgmf_balanced_cuts": ([I64, I64, I32, vp, vp, I64, I64, I64, vp, vp], c_int),
        "bgmf_reorder_ids": ([I64, I64, I32, vp, vp, I64, vp, vp], c_int),
        "bgmf_query_sizes": ([vp, I64, ctypes.POINTER(ctypes.c_size_t),
                              ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_size_t),
                              ctypes.POINTER(ctypes.c_size_t)], c_int),
        "bgmf_bind": ([vp, vp, vp, vp, ctypes.c_size_t, vp, ctypes.c_size_t, vp], c_int),
    }
    for name, (args, res) in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = res
    return lib


_lib = _load()


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def _check(h, rc: int):
    if rc != BGMF_OK:
        msg = _lib.bgmf_last_error(h)
        raise BgmfError(rc, msg.decode() if msg else "")


# --- functions with the C names (argument marshalling only) -----------------

def bgmf_create(n: int, m: int, k: int, p: int):
    h = _lib.bgmf_create(int(n), int(m), int(k), int(p))
    if not h:
        msg = _lib.bgmf_last_error(None)
        raise BgmfError(BGMF_E_ARG, msg.decode() if msg else "bgmf_create failed")
    return h


def bgmf_destroy(h) -> None:
    _lib.bgmf_destroy(h)


def bgmf_last_error(h) -> str:
    msg = _lib.bgmf_last_error(h)
    return msg.decode() if msg else ""


def bgmf_set_stream(h, stream) -> None:
    """``stream``: an integer hipStream_t (e.g. torch.cuda.current_stream().cuda_stream)
    or None for the handle's own stream."""
    _check(h, _lib.bgmf_set_stream(h, ctypes.c_void_p(int(stream)) if stream else None))


def bgmf_query_sizes(h, nnz: int):
    """Returns dict(factor_bytes, min_ws_bytes, incore_ws_bytes, pinned_bytes)."""
    out = [ctypes.c_size_t(0) for _ in range(4)]
    _check(h, _lib.bgmf_query_sizes(h, int(nnz), *[ctypes.byref(o) for o in out]))
    keys = ("factor_bytes", "min_ws_bytes", "incore_ws_bytes", "pinned_bytes")
    return {k: int(o.value) for k, o in zip(keys, out)}


def bgmf_bind(h, U_dev: int, V_dev: int, ws_dev: int, ws_bytes: int, pinned_host: int,
              pinned_bytes: int, stream) -> None:
    """Addresses as integers (for example ``tensor.data_ptr()``), ``pinned_host``
    0 for none, ``stream`` an integer hipStream_t or None."""
    def vp(x):
        return ctypes.c_void_p(int(x)) if x else None
    _check(h, _lib.bgmf_bind(h, vp(U_dev), vp(V_dev), vp(ws_dev), int(ws_bytes),
                             vp(pinned_host), int(pinned_bytes), vp(stream)))


def bgmf_set_factors(h, U: np.ndarray, V: np.ndarray) -> None:
    U = np.ascontiguousarray(U, dtype=np.float32)
    V = np.ascontiguousarray(V, dtype=np.float32)
    _check(h, _lib.bgmf_set_factors(h, _ptr(U), _ptr(V)))


def bgmf_load_coo(h, rows, cols, vals) -> None:
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    cols = np.ascontiguousarray(cols, dtype=np.int32)
    vals = np.ascontiguousarray(vals, dtype=np.float32)
    if not (rows.shape == cols.shape == vals.shape and rows.ndim == 1):
        raise ValueError("rows, cols and vals must be 1-D arrays of one length")
    _check(h, _lib.bgmf_load_coo(h, _ptr(rows), _ptr(cols), _ptr(vals), rows.shape[0]))


def bgmf_epoch(h, alpha: float, beta: float) -> None:
    _check(h, _lib.bgmf_epoch(h, float(alpha), float(beta)))


def bgmf_rmse(h) -> float:
    out = ctypes.c_double(math.nan)
    _check(h, _lib.bgmf_rmse(h, ctypes.byref(out)))
    return out.value


def bgmf_get_factors(h, n: int, m: int, k: int):
    U = np.empty((n, k), dtype=np.float32)
    V = np.empty((m, k), dtype=np.float32)
    _check(h, _lib.bgmf_get_factors(h, _ptr(U), _ptr(V)))
    return U, V


def bgmf_get_layout(h, p: int, nnz: int):
    block_ptr = np.empty(p * p + 1, dtype=np.int64)
    perm = np.empty(max(nnz, 1), dtype=np.int32)
    _check(h, _lib.bgmf_get_layout(h, _ptr(block_ptr), _ptr(perm)))
    return block_ptr, perm[:nnz]


def bgmf_sync(h) -> None:
    _check(h, _lib.bgmf_sync(h))


def bgmf_factor_ptrs(h):
    u, v = ctypes.c_void_p(), ctypes.c_void_p()
    _check(h, _lib.bgmf_factor_ptrs(h, ctypes.byref(u), ctypes.byref(v)))
    return u.value, v.value


def bgmf_set_option(h, option: int, value: int) -> None:
    _check(h, _lib.bgmf_set_option(h, int(option), int(value)))


def bgmf_get_option(h, option: int) -> int:
    out = ctypes.c_int64()
    _check(h, _lib.bgmf_get_option(h, int(option), ctypes.byref(out)))
    return out.value


def bgmf_get_timing(h):
    e, r = ctypes.c_double(), ctypes.c_double()
    _check(h, _lib.bgmf_get_timing(h, ctypes.byref(e), ctypes.byref(r)))
    return e.value, r.value


def bgmf_chain_stats(h):
    out = np.zeros(4, dtype=np.int64)
    _check(h, _lib.bgmf_chain_stats(h, _ptr(out)))
    return out


def bgmf_get_trace(h, p: int):
    """Block trace of the last epoch: (begin, end, ticks_per_s), begin and end
    as [p, p] arrays indexed [s, b] (slot s*p + b)."""
    begin = np.zeros(p * p, dtype=np.int64)
    end = np.zeros(p * p, dtype=np.int64)
    tps = ctypes.c_int64(0)
    _check(h, _lib.bgmf_get_trace(h, _ptr(begin), _ptr(end), ctypes.byref(tps)))
    return begin.reshape(p, p), end.reshape(p, p), int(tps.value)


def bgmf_rmse_coo(h, rows, cols, vals) -> float:
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    cols = np.ascontiguousarray(cols, dtype=np.int32)
    vals = np.ascontiguousarray(vals, dtype=np.float32)
    if not (rows.shape == cols.shape == vals.shape and rows.ndim == 1):
        raise ValueError("rows, cols and vals must be 1-D arrays of one length")
    out = ctypes.c_double(math.nan)
    _check(h, _lib.bgmf_rmse_coo(h, _ptr(rows), _ptr(cols), _ptr(vals), rows.shape[0],
                                 ctypes.byref(out)))
    return out.value


def bgmf_rmse_coo_dev(h, rows_dev: int, cols_dev: int, vals_dev: int, nnz: int) -> float:
    """Device addresses as integers (for example ``tensor.data_ptr()``)."""
    out = ctypes.c_double(math.nan)
    _check(h, _lib.bgmf_rmse_coo_dev(h, ctypes.c_void_p(int(rows_dev)),
                                     ctypes.c_void_p(int(cols_dev)),
                                     ctypes.c_void_p(int(vals_dev)), int(nnz),
                                     ctypes.byref(out)))
    return out.value


def bgmf_fit(h, alpha: float, beta: float, max_epochs: int, delta: float):
    """Returns (epochs_run, rmse_history[: epochs_run + 1])."""
    hist = np.full(int(max_epochs) + 1, np.nan, dtype=np.float64)
    ran = ctypes.c_int32(0)
    rc = _lib.bgmf_fit(h, float(alpha), float(beta), int(max_epochs), float(delta),
                       ctypes.byref(ran), _ptr(hist))
    if rc != BGMF_OK:
        msg = _lib.bgmf_last_error(h)
        err = BgmfError(rc, msg.decode() if msg else "")
        err.epochs_run, err.rmse_history = ran.value, hist[: ran.value + 1]
        raise err
    return ran.value, hist[: ran.value + 1]


def bgmf_set_cuts(h, row_cuts, col_cuts) -> None:
    r = np.ascontiguousarray(row_cuts, dtype=np.int64)
    c = np.ascontiguousarray(col_cuts, dtype=np.int64)
    _check(h, _lib.bgmf_set_cuts(h, _ptr(r), _ptr(c)))


def bgmf_get_cuts(h, p: int):
    r = np.empty(p + 1, dtype=np.int64)
    c = np.empty(p + 1, dtype=np.int64)
    _check(h, _lib.bgmf_get_cuts(h, _ptr(r), _ptr(c)))
    return r, c


def bgmf_balanced_cuts(n: int, m: int, p: int, rows, cols, max_rows: int = 65536,
                       max_cols: int = 65536):
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    cols = np.ascontiguousarray(cols, dtype=np.int32)
    r = np.empty(p + 1, dtype=np.int64)
    c = np.empty(p + 1, dtype=np.int64)
    rc = _lib.bgmf_balanced_cuts(int(n), int(m), int(p), _ptr(rows), _ptr(cols), rows.shape[0],
                                 int(max_rows), int(max_cols), _ptr(r), _ptr(c))
    if rc != BGMF_OK:
        msg = _lib.bgmf_last_error(None)
        raise BgmfError(rc, msg.decode() if msg else "bgmf_balanced_cuts failed")
    return r, c


def bgmf_reorder_ids(n: int, m: int, p: int, rows, cols):
    """Returns (row_newid[n], col_newid[m]) as int32 arrays."""
    rows = np.ascontiguousarray(rows, dtype=np.int32)
    cols = np.ascontiguousarray(cols, dtype=np.int32)
    rn = np.empty(int(n), dtype=np.int32)
    cn = np.empty(int(m), dtype=np.int32)
    rc = _lib.bgmf_reorder_ids(int(n), int(m), int(p), _ptr(rows), _ptr(cols), rows.shape[0],
                               _ptr(rn), _ptr(cn))
    if rc != BGMF_OK:
        msg = _lib.bgmf_last_error(None)
        raise BgmfError(rc, msg.decode() if msg else "bgmf_reorder_ids failed")
    return rn, cn


# --- convenience wrapper -----------------------------------------------------

class Model:
    """Owns one handle: ``Model(n, m, k, p)``; see include/bgmf.h."""

    def __init__(self, n: int, m: int, k: int, p: int):
        self.n, self.m, self.k, self.p = int(n), int(m), int(k), int(p)
        self.nnz = 0
        self.h = bgmf_create(n, m, k, p)

    def close(self):
        if self.h:
            bgmf_destroy(self.h)
            self.h = None

    def __del__(self):
        # at interpreter shutdown the HIP runtime may already be torn down:
        # leave the handle to the process exit instead of calling into it
        if sys.is_finalizing():
            return
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def set_stream(self, stream):
        bgmf_set_stream(self.h, stream)

    def set_factors(self, U, V):
        bgmf_set_factors(self.h, U, V)

    def query_sizes(self, nnz: int):
        return bgmf_query_sizes(self.h, nnz)

    def bind(self, U_dev: int, V_dev: int, ws_dev: int, ws_bytes: int, pinned_host: int = 0,
             pinned_bytes: int = 0, stream=None):
        bgmf_bind(self.h, U_dev, V_dev, ws_dev, ws_bytes, pinned_host, pinned_bytes, stream)

    def bind_tensors(self, U, V, ws, pinned=None, stream=None):
        """bind() with tensors (anything with data_ptr(), numel() and
        element_size(), such as torch tensors): U (n x k) and V (m x k) float32
        on the device, ws a device byte buffer, pinned a pinned host byte
        buffer or None, stream an integer hipStream_t or None."""
        def nbytes(t):
            return int(t.numel()) * int(t.element_size())
        for t, rows in ((U, self.n), (V, self.m)):
            if nbytes(t) != rows * self.k * 4:
                raise ValueError("U must hold n x k and V m x k float32 values")
        bgmf_bind(self.h, U.data_ptr(), V.data_ptr(), ws.data_ptr(), nbytes(ws),
                  pinned.data_ptr() if pinned is not None else 0,
                  nbytes(pinned) if pinned is not None else 0, stream)

    def load_coo(self, rows, cols, vals):
        bgmf_load_coo(self.h, rows, cols, vals)
        self.nnz = int(np.asarray(rows).shape[0])

    def epoch(self, alpha: float, beta: float):
        bgmf_epoch(self.h, alpha, beta)

    def rmse(self) -> float:
        return bgmf_rmse(self.h)

    def get_factors(self):
        return bgmf_get_factors(self.h, self.n, self.m, self.k)

    def get_layout(self):
        return bgmf_get_layout(self.h, self.p, self.nnz)

    def sync(self):
        bgmf_sync(self.h)

    def set_option(self, option: int, value: int):
        bgmf_set_option(self.h, option, value)

    def get_option(self, option: int) -> int:
        return bgmf_get_option(self.h, option)

    def timing(self):
        return bgmf_get_timing(self.h)

    def chain_stats(self):
        return bgmf_chain_stats(self.h)

    def get_trace(self):
        return bgmf_get_trace(self.h, self.p)

    def rmse_coo(self, rows, cols, vals) -> float:
        return bgmf_rmse_coo(self.h, rows, cols, vals)

    def fit(self, alpha: float, beta: float, max_epochs: int, delta: float):
        return bgmf_fit(self.h, alpha, beta, max_epochs, delta)

    def set_cuts(self, row_cuts, col_cuts):
        bgmf_set_cuts(self.h, row_cuts, col_cuts)

    def get_cuts(self):
        return bgmf_get_cuts(self.h, self.p)
