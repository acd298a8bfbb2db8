"""CPU oracle for blocked SGD matrix factorisation — TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the benchmark's
``cpu_baseline`` leg may import this package.  The HIP library and its Python
binding never import, link or call it; the two share no code.

The arithmetic lives in ``bgmf_oracle.c`` (plain C, fp32 with every operation
rounded separately, ``-ffp-contract=off``); this module only compiles it with
gcc and marshals numpy arrays through ctypes.  ``pyoracle`` is an independent
pure-Python twin for tiny inputs.

Functions follow the paper's Section 1:
  * ``bucket``   — the p x p block grid of Eq. 4 and the strata of Section 1.1
  * ``bucket_cuts`` — the same with given (unequal) block boundaries
  * ``sgd_update`` — one per-rating step of Eq. 2-3 (Eq. 14-15 per element)
  * ``epoch`` / ``epoch_mt`` / ``epoch_ordered`` — one CPU step of
    Algorithm 1 with one pass per block
  * ``epoch_passes`` — the same with GPU_STEPS passes per block
  * ``rmse``     — whole-matrix RMSE used by Algorithm 1's termination test
  * ``loss``     — the objective of Eq. 1 (fp64)
  * ``sgd_update_f64`` / ``epoch_f64`` — the same step and epoch carried out
    in binary64, the exact-arithmetic reference for measuring how far the
    binary32 schedule (the oracle's or the GPU's) drifts through rounding
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "bgmf_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_CFLAGS = ["-O2", "-ffp-contract=off", "-fno-fast-math", "-fno-unsafe-math-optimizations",
           "-Wall", "-shared", "-fPIC", "-pthread"]


def build(force: bool = True) -> str:
    """Compile the C oracle with gcc into ``oracle/liboracle.so``."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.run(["gcc", *_CFLAGS, _SRC, "-o", tmp, "-lm"], check=True)
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        i32p = np.ctypeslib.ndpointer(np.int32, flags="C_CONTIGUOUS")
        i64p = np.ctypeslib.ndpointer(np.int64, flags="C_CONTIGUOUS")
        f32p = np.ctypeslib.ndpointer(np.float32, flags="C_CONTIGUOUS")
        f64p = np.ctypeslib.ndpointer(np.float64, flags="C_CONTIGUOUS")
        I64, I32, F32, F64 = ctypes.c_int64, ctypes.c_int32, ctypes.c_float, ctypes.c_double
        lib.oracle_bucket.argtypes = [I64, I64, I64, I64, i32p, i32p, i64p, i32p]
        lib.oracle_bucket.restype = ctypes.c_int
        lib.oracle_bucket_cuts.argtypes = [I64, I64, I64, i64p, i64p, I64, i32p, i32p, i64p, i32p]
        lib.oracle_bucket_cuts.restype = ctypes.c_int
        lib.oracle_sgd_update.argtypes = [I32, f32p, f32p, F32, F32, F32]
        lib.oracle_sgd_update.restype = None
        lib.oracle_sgd_update_f64.argtypes = [I32, f64p, f64p, F32, F32, F32]
        lib.oracle_sgd_update_f64.restype = None
        lib.oracle_epoch.argtypes = [I64, I32, i32p, i32p, f32p, i64p, i32p, f32p, f32p, F32, F32]
        lib.oracle_epoch.restype = None
        lib.oracle_epoch_ordered.argtypes = [I64, I32, i32p, i32p, f32p, i64p, i32p, f32p, f32p,
                                             F32, F32, i32p]
        lib.oracle_epoch_ordered.restype = None
        lib.oracle_epoch_mt.argtypes = [I64, I32, i32p, i32p, f32p, i64p, i32p, f32p, f32p,
                                        F32, F32, I32]
        lib.oracle_epoch_mt.restype = ctypes.c_int
        lib.oracle_epoch_mt_f64.argtypes = [I64, I32, i32p, i32p, f32p, i64p, i32p, f64p, f64p,
                                            F32, F32, I32]
        lib.oracle_epoch_mt_f64.restype = ctypes.c_int
        lib.oracle_epoch_passes.argtypes = [I64, I32, i32p, i32p, f32p, i64p, i32p, f32p, f32p,
                                            F32, F32, I32]
        lib.oracle_epoch_passes.restype = None
        lib.oracle_epoch_mt_passes.argtypes = [I64, I32, i32p, i32p, f32p, i64p, i32p, f32p,
                                               f32p, F32, F32, I32, I32]
        lib.oracle_epoch_mt_passes.restype = ctypes.c_int
        lib.oracle_rmse.argtypes = [I32, I64, i32p, i32p, f32p, f32p, f32p]
        lib.oracle_rmse.restype = F64
        lib.oracle_loss.argtypes = [I32, I64, i32p, i32p, f32p, f32p, f32p, F64]
        lib.oracle_loss.restype = F64
        _lib = lib
    return _lib


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def bucket(n: int, m: int, p: int, rows, cols):
    """Return ``(block_ptr[p*p+1] int64, perm[nnz] int32)``."""
    rows = _c(rows, np.int32)
    cols = _c(cols, np.int32)
    nnz = rows.shape[0]
    block_ptr = np.zeros(p * p + 1, dtype=np.int64)
    perm = np.zeros(max(nnz, 1), dtype=np.int32)
    rc = _load().oracle_bucket(n, m, p, nnz, rows, cols, block_ptr, perm)
    if rc != 0:
        raise MemoryError("oracle_bucket: out of memory")
    return block_ptr, perm[:nnz]


def bucket_cuts(n: int, m: int, p: int, row_cuts, col_cuts, rows, cols):
    """Bucketing with given block boundaries (p + 1 cut points per
    dimension); returns (block_ptr, perm) as ``bucket``."""
    rows = _c(rows, np.int32)
    cols = _c(cols, np.int32)
    nnz = rows.shape[0]
    bp = np.zeros(p * p + 1, dtype=np.int64)
    perm = np.zeros(max(nnz, 1), dtype=np.int32)
    rc = _load().oracle_bucket_cuts(n, m, p, _c(row_cuts, np.int64), _c(col_cuts, np.int64), nnz,
                                    rows, cols, bp, perm)
    if rc != 0:
        raise MemoryError("oracle_bucket_cuts: out of memory")
    return bp, perm[:nnz]


def sgd_update(u, v, x: float, alpha: float, beta: float):
    """One step of Eq. 2-3 on copies of u, v; returns (u', v')."""
    u = _c(u, np.float32).copy()
    v = _c(v, np.float32).copy()
    _load().oracle_sgd_update(u.shape[0], u, v, float(x), float(alpha), float(beta))
    return u, v


def _epoch_args(p, rows, cols, vals, block_ptr, perm, U, V):
    U = _c(U, np.float32)
    V = _c(V, np.float32)
    perm = _c(perm, np.int32)
    if perm.shape[0] == 0:
        perm = np.zeros(1, dtype=np.int32)
    return (int(p), int(U.shape[1]), _c(rows, np.int32), _c(cols, np.int32), _c(vals, np.float32),
            _c(block_ptr, np.int64), perm, U, V)


def epoch(p, rows, cols, vals, block_ptr, perm, U, V, alpha, beta):
    """One blocked SGD epoch, in place on U and V (fp32, row-major)."""
    args = _epoch_args(p, rows, cols, vals, block_ptr, perm, U, V)
    assert args[7] is U and args[8] is V, "U and V must be C-contiguous float32 (updated in place)"
    _load().oracle_epoch(*args, float(alpha), float(beta))


def epoch_ordered(p, rows, cols, vals, block_ptr, perm, U, V, alpha, beta, order):
    """As ``epoch`` with the blocks of stratum s visited as order[s*p + idx]."""
    args = _epoch_args(p, rows, cols, vals, block_ptr, perm, U, V)
    assert args[7] is U and args[8] is V
    _load().oracle_epoch_ordered(*args, float(alpha), float(beta), _c(order, np.int32))


def epoch_mt(p, rows, cols, vals, block_ptr, perm, U, V, alpha, beta, threads):
    """Multithreaded epoch (blocks of a stratum over threads); returns threads used."""
    args = _epoch_args(p, rows, cols, vals, block_ptr, perm, U, V)
    assert args[7] is U and args[8] is V
    return int(_load().oracle_epoch_mt(*args, float(alpha), float(beta), int(threads)))


def epoch_passes(p, rows, cols, vals, block_ptr, perm, U, V, alpha, beta, passes, threads=1):
    """One epoch with GPU_STEPS = ``passes`` (Algorithm 1, Section 1.3): every
    block swept ``passes`` times in a row before the next; in place on U, V;
    returns threads used."""
    args = _epoch_args(p, rows, cols, vals, block_ptr, perm, U, V)
    assert args[7] is U and args[8] is V
    if threads <= 1:
        _load().oracle_epoch_passes(*args, float(alpha), float(beta), int(passes))
        return 1
    return int(_load().oracle_epoch_mt_passes(*args, float(alpha), float(beta), int(passes),
                                              int(threads)))


def sgd_update_f64(u, v, x: float, alpha: float, beta: float):
    """One step of Eq. 2-3 in binary64 on copies of u, v (x, alpha, beta
    are rounded to binary32 first, as the GPU receives them)."""
    u = _c(u, np.float64).copy()
    v = _c(v, np.float64).copy()
    _load().oracle_sgd_update_f64(u.shape[0], u, v, float(x), float(alpha), float(beta))
    return u, v


def epoch_f64(p, rows, cols, vals, block_ptr, perm, U64, V64, alpha, beta, threads=1):
    """The epoch in binary64, in place on float64 U64 and V64: the same
    schedule and operation order as ``epoch``, as an exact-arithmetic
    reference for measuring binary32 rounding; returns threads used."""
    args = list(_epoch_args(p, rows, cols, vals, block_ptr, perm, np.zeros((1, 1), np.float32),
                            np.zeros((1, 1), np.float32)))
    U64 = _c(U64, np.float64)
    V64 = _c(V64, np.float64)
    args[1] = int(U64.shape[1])
    args[7], args[8] = U64, V64
    return int(_load().oracle_epoch_mt_f64(*args, float(alpha), float(beta), int(threads)))


def rmse(rows, cols, vals, U, V) -> float:
    U = _c(U, np.float32)
    V = _c(V, np.float32)
    rows = _c(rows, np.int32)
    return float(_load().oracle_rmse(U.shape[1], rows.shape[0], rows, _c(cols, np.int32),
                                     _c(vals, np.float32), U, V))


def loss(rows, cols, vals, U, V, beta: float) -> float:
    U = _c(U, np.float32)
    V = _c(V, np.float32)
    rows = _c(rows, np.int32)
    return float(_load().oracle_loss(U.shape[1], rows.shape[0], rows, _c(cols, np.int32),
                                     _c(vals, np.float32), U, V, float(beta)))
