"""Synthetic rating matrices with the shapes of the benchmark workloads.

Every array is drawn from seeded generators (numpy's PCG64, and per-index
SplitMix64 streams in gen.c), so a workload is a pure function of its
parameters, independent of the thread count.  Nothing here updates factors or evaluates
the method; the planted low-rank model below only produces rating VALUES.

Recipes (the public rating datasets the paper evaluates on are not
available; these stand in for them):

* ``uniform``   — ``nnz`` distinct cells drawn uniformly without replacement
  from the n x m grid (tiny config).
* ``powerlaw``  — a bipartite graph with heavy-tailed degrees.  Each user i
  gets a degree d_i (``user_deg``: Zipf weights rank^-a on a seeded
  permutation of user ids, or a lognormal with a given median), rescaled so
  the degrees sum to exactly ``nnz`` and clipped to [1, m].  User i then
  draws d_i DISTINCT items by successive sampling without replacement from
  Zipf(a_item) item weights placed on a seeded permutation of item ids (the
  C helper in gen.c).  The most popular items saturate at n raters.
* ``dense``     — every cell of the n x m grid (the paper's Table 1 shape).

Values:
* ``int5``    — x = clip(rint(c + u*.v* + eps), 1, 5) with a planted rank-r
  model u*, v* ~ N(0, 1/sqrt(r)) entrywise, eps ~ N(0, noise), and c chosen
  so the mean of c + u*.v* over observed cells is 3.
* ``cont100`` — x = clip(50 + 20 z + eps, 0, 100), z = u*.v* scaled to unit
  standard deviation over observed cells, eps ~ N(0, noise).
* ``uint``    — integers uniform in [lo, hi] (Table 1's pseudo-random matrix).

The COO order is a seeded shuffle (seed ``seed_order``); the initial factors
are U(0, 0.1) drawn in float64 (seed ``seed_init``) and rounded to float32.
"""
from __future__ import annotations

import dataclasses
import hashlib
import json
import os
import subprocess
import ctypes
from typing import Optional

import numpy as np


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n: int
    m: int
    k: int
    p: int
    alpha: float
    beta: float
    epochs: int
    rows: np.ndarray  # int32[nnz]
    cols: np.ndarray  # int32[nnz]
    vals: np.ndarray  # float32[nnz]
    U0: np.ndarray    # float32[n, k]
    V0: np.ndarray    # float32[m, k]
    planted: Optional[np.ndarray] = None  # float32[nnz] noiseless planted prediction, if kept

    @property
    def nnz(self) -> int:
        return int(self.rows.shape[0])


# Parameters of the five benchmark workloads (sizes, degree structure, value
# model, factor width k, grid p, step sizes, epochs, seeds) and of the
# paper's Table 1 matrix.  The 250M-rating workload's stated step 0.002 makes
# sequential SGD diverge on it (ratings in [0, 100], k = 128), so it runs at
# 5e-4, the largest step tried at which the exact epoch stays finite.  The "ooc" workload is meant to be run with its
# ratings streamed from host memory under OOC_BUDGET_BYTES of device memory.
CONFIGS = {
    "tiny": dict(n=2_000, m=1_000, nnz=100_000, structure="uniform", values="int5", rank=8,
                 noise=0.5, k=16, p=4, alpha=0.01, beta=0.05, epochs=5, seed=1),
    "medium": dict(n=70_000, m=10_000, nnz=10_000_000, structure="powerlaw",
                   user_deg=("zipf", 1.0), item_zipf=1.1, values="int5", rank=16, noise=0.5,
                   k=32, p=256, alpha=0.01, beta=0.05, epochs=20, seed=2),
    "large": dict(n=480_000, m=18_000, nnz=100_000_000, structure="powerlaw",
                  user_deg=("lognormal", 100.0, 1.2116), item_zipf=1.2, values="int5", rank=32,
                  noise=0.5, k=64, p=1024, alpha=0.005, beta=0.05, epochs=20, seed=3),
    "vlarge": dict(n=1_000_000, m=625_000, nnz=250_000_000, structure="powerlaw",
                   user_deg=("zipf", 1.1), item_zipf=1.1, values="cont100", rank=64, noise=5.0,
                   k=128, p=2048, alpha=5e-4, beta=0.02, epochs=10, seed=4),
    "ooc": dict(n=10_000_000, m=5_000_000, nnz=2_000_000_000, structure="powerlaw",
                user_deg=("zipf", 1.1), item_zipf=1.1, values="int5", rank=32, noise=0.5,
                k=64, p=4096, alpha=0.005, beta=0.05, epochs=3, seed=5),
    "table1": dict(n=1024, m=1024, nnz=1024 * 1024, structure="dense", values="uint", lo=1, hi=30,
                   k=16, p=32, alpha=2e-4, beta=5e-3, epochs=6, seed=6),
}


OOC_BUDGET_BYTES = 16_000_000_000


def _zipf_weights(count: int, a: float) -> np.ndarray:
    return np.arange(1, count + 1, dtype=np.float64) ** (-a)


def _scale_to_total(raw: np.ndarray, total: int, cap: int) -> np.ndarray:
    """Integer degrees >= 1, <= cap, proportional to raw, summing to total."""
    raw = np.asarray(raw, dtype=np.float64)
    scale = total / raw.sum()
    for _ in range(100):
        d = np.clip(np.rint(raw * scale), 1, cap)
        s = d.sum()
        if abs(s - total) <= max(1, total // 100000):
            break
        free = d < cap
        scale *= 1.0 + (total - s) / max(1.0, float((raw * scale)[free].sum()))
    d = d.astype(np.int64)
    diff = int(total - d.sum())
    # settle the last few units on uncapped / above-one users in a fixed order
    order = np.argsort(-raw, kind="stable")
    idx = 0
    while diff != 0 and idx < 10 * len(order):
        u = order[idx % len(order)]
        if diff > 0 and d[u] < cap:
            d[u] += 1
            diff -= 1
        elif diff < 0 and d[u] > 1:
            d[u] -= 1
            diff += 1
        idx += 1
    return d


def _user_degrees(rng, n, m, nnz, spec) -> np.ndarray:
    kind = spec[0]
    if kind == "zipf":
        raw = _zipf_weights(n, spec[1])
        raw = raw[rng.permutation(n)]  # rank -> user id
    elif kind == "lognormal":
        median, sigma = spec[1], spec[2]
        raw = rng.lognormal(mean=np.log(median), sigma=sigma, size=n)
    else:
        raise ValueError(kind)
    return _scale_to_total(raw, min(nnz, n * m), m)


def _powerlaw_cells(rng, n, m, nnz, user_deg, item_zipf, seed):
    """Return (rows, cols) of ``nnz`` distinct cells, grouped by user."""
    deg = _user_degrees(rng, n, m, nnz, user_deg)
    w_item = _zipf_weights(m, item_zipf)
    item_of_rank = rng.permutation(m).astype(np.int32)
    cdf_item = np.cumsum(w_item)
    cdf_item /= cdf_item[-1]
    offset = np.zeros(n, dtype=np.int64)
    np.cumsum(deg[:-1], out=offset[1:])
    total = int(deg.sum())
    cols = np.empty(total, dtype=np.int32)
    lib = _genlib()
    rc = lib.gen_user_items(n, m, _ptr(deg), _ptr(offset), _ptr(cdf_item), _ptr(w_item),
                            _ptr(item_of_rank), ctypes.c_uint64(seed * 7919 + 17), _ptr(cols))
    if rc != 0:
        raise MemoryError("gen_user_items failed")
    rows = np.repeat(np.arange(n, dtype=np.int32), deg)
    return rows, cols


def _planted_dot(rng, rows, cols, n, m, rank):
    us = (rng.standard_normal((n, rank)) / np.sqrt(rank)).astype(np.float32)
    vs = (rng.standard_normal((m, rank)) / np.sqrt(rank)).astype(np.float32)
    z = np.empty(rows.shape[0], dtype=np.float64)
    _genlib().gen_planted_dot(rows.shape[0], rank, _ptr(rows), _ptr(cols), _ptr(us), _ptr(vs),
                              _ptr(z))
    return z


def _normal(count, seed):
    out = np.empty(count, dtype=np.float64)
    _genlib().gen_normal(count, ctypes.c_uint64(seed), _ptr(out))
    return out


def _permutation(count, seed):
    """Seeded uniform permutation of 0..count-1 (int64), the same for any
    thread count (see gen_permutation in gen.c)."""
    out = np.empty(count, dtype=np.int64)
    if _genlib().gen_permutation(count, ctypes.c_uint64(seed * 2654435761 + 11), _ptr(out)) != 0:
        raise MemoryError("gen_permutation failed")
    return out


def _gather(order, a):
    """a[order] for a 4-byte array, in parallel."""
    assert a.dtype.itemsize == 4
    out = np.empty_like(a)
    _genlib().gen_gather32(a.shape[0], _ptr(order), _ptr(np.ascontiguousarray(a)), _ptr(out))
    return out


_GEN = None
_HERE = os.path.dirname(os.path.abspath(__file__))


def build(force: bool = True) -> str:
    """Compile the generator helper (gcc, OpenMP) into workloads/libgen.so."""
    src = os.path.join(_HERE, "gen.c")
    lib = os.path.join(_HERE, "libgen.so")
    if force or not os.path.exists(lib) or os.path.getmtime(lib) < os.path.getmtime(src):
        tmp = lib + ".tmp"
        subprocess.run(["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-Wall", src, "-o", tmp,
                        "-lm"], check=True)
        os.replace(tmp, lib)
    return lib


def _genlib():
    global _GEN
    if _GEN is None:
        lib = ctypes.CDLL(build(force=False))
        vp = ctypes.c_void_p
        I64 = ctypes.c_int64
        lib.gen_user_items.argtypes = [I64, I64, vp, vp, vp, vp, vp, ctypes.c_uint64, vp]
        lib.gen_user_items.restype = ctypes.c_int
        lib.gen_planted_dot.argtypes = [I64, ctypes.c_int32, vp, vp, vp, vp, vp]
        lib.gen_planted_dot.restype = None
        lib.gen_normal.argtypes = [I64, ctypes.c_uint64, vp]
        lib.gen_normal.restype = None
        lib.gen_permutation.argtypes = [I64, ctypes.c_uint64, vp]
        lib.gen_permutation.restype = ctypes.c_int
        lib.gen_gather32.argtypes = [I64, vp, vp, vp]
        lib.gen_gather32.restype = None
        _GEN = lib
    return _GEN


def _ptr(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


def make(name: str, n: int, m: int, nnz: int, k: int, p: int, alpha: float, beta: float,
         epochs: int, seed: int, structure: str, values: str, rank: int = 8, noise: float = 0.5,
         user_deg=("zipf", 1.0), item_zipf: float = 1.1, lo: int = 1, hi: int = 30,
         seed_init: Optional[int] = None, seed_order: Optional[int] = None,
         cache_dir: Optional[str] = None, keep_planted: bool = False,
         log=None) -> Workload:
    """Draw one workload.  Seeds: data ``seed``; init ``seed_init`` (default
    100 + seed); order shuffle ``seed_order`` (default 200 + seed).  With
    ``keep_planted`` the noiseless planted prediction of every rating is kept
    (in COO order) for noise-floor estimates.  ``log``, if given, is called
    with a short message after each generation phase."""
    seed_init = 100 + seed if seed_init is None else seed_init
    seed_order = 200 + seed if seed_order is None else seed_order
    params = dict(n=n, m=m, nnz=nnz, k=k, p=p, seed=seed, structure=structure, values=values,
                  rank=rank, noise=noise, user_deg=list(user_deg), item_zipf=item_zipf, lo=lo,
                  hi=hi, seed_init=seed_init, seed_order=seed_order, version=4)
    tag = hashlib.sha1(json.dumps(params, sort_keys=True).encode()).hexdigest()[:16]
    cache_dir = cache_dir or os.environ.get("BGMF_WORKLOAD_CACHE")
    arrays = _load_cache(cache_dir, tag) if cache_dir else None
    if arrays is None:
        arrays = _draw(n, m, nnz, k, seed, structure, values, rank, noise, user_deg, item_zipf,
                       lo, hi, seed_init, seed_order, log or (lambda msg: None))
        if cache_dir:
            _save_cache(cache_dir, tag, arrays)
    rows, cols, vals, U0, V0, planted = arrays
    return Workload(name, n, m, k, p, alpha, beta, epochs, rows, cols, vals, U0, V0,
                    planted if keep_planted else None)


def _draw(n, m, nnz, k, seed, structure, values, rank, noise, user_deg, item_zipf, lo, hi,
          seed_init, seed_order, log):
    rng = np.random.Generator(np.random.PCG64(seed))
    if structure == "uniform":
        if nnz > n * m:
            raise ValueError("nnz exceeds n*m")
        cells = rng.choice(n * m, size=nnz, replace=False).astype(np.int64)
    elif structure == "dense":
        cells = np.arange(n * m, dtype=np.int64)
        nnz = n * m
    elif structure == "powerlaw":
        cells = None
        rows, cols = _powerlaw_cells(rng, n, m, nnz, tuple(user_deg), item_zipf, seed)
    else:
        raise ValueError(structure)
    if cells is not None:
        rows = (cells // m).astype(np.int32)
        cols = (cells % m).astype(np.int32)
        del cells
    log(f"cells drawn: {rows.shape[0]}")

    if values == "int5":
        z = _planted_dot(rng, rows, cols, n, m, rank)
        z += 3.0 - z.mean()
        planted = z.astype(np.float32)
        z += noise * _normal(z.shape[0], seed * 104729 + 3)
        vals = np.clip(np.rint(z), 1.0, 5.0).astype(np.float32)
    elif values == "cont100":
        z = _planted_dot(rng, rows, cols, n, m, rank)
        z = 50.0 + 20.0 * (z - z.mean()) / max(z.std(), 1e-12)
        planted = z.astype(np.float32)
        z += noise * _normal(z.shape[0], seed * 104729 + 3)
        vals = np.clip(z, 0.0, 100.0).astype(np.float32)
    elif values == "uint":
        vals = rng.integers(lo, hi + 1, size=rows.shape[0]).astype(np.float32)
        planted = np.full(rows.shape[0], 0.5 * (lo + hi), dtype=np.float32)
    else:
        raise ValueError(values)
    z = None
    log("values drawn")

    order = _permutation(rows.shape[0], seed_order)
    log("order drawn")
    rows, cols, vals, planted = (_gather(order, a) for a in (rows, cols, vals, planted))
    del order
    log("ratings shuffled")
    U0, V0 = init_factors(n, m, k, seed_init)
    return (np.ascontiguousarray(rows), np.ascontiguousarray(cols), np.ascontiguousarray(vals),
            U0, V0, np.ascontiguousarray(planted))


def init_factors(n: int, m: int, k: int, seed: int, lo: float = 0.0, hi: float = 0.1):
    """U(lo, hi) initial factors, drawn in float64 and rounded to float32."""
    rng = np.random.Generator(np.random.PCG64(seed))
    U0 = rng.uniform(lo, hi, size=(n, k)).astype(np.float32)
    V0 = rng.uniform(lo, hi, size=(m, k)).astype(np.float32)
    return U0, V0


def make_config(name: str, cache_dir: Optional[str] = None, **overrides) -> Workload:
    """One of the named workloads, optionally with parameters overridden
    (for example a smaller nnz with the same structure)."""
    params = dict(CONFIGS[name])
    params.update(overrides)
    return make(name, cache_dir=cache_dir, **params)


_NAMES = ("rows", "cols", "vals", "U0", "V0", "planted")


def _load_cache(cache_dir, tag):
    paths = [os.path.join(cache_dir, f"{tag}_{nm}.npy") for nm in _NAMES]
    if not all(os.path.exists(pth) for pth in paths):
        return None
    return tuple(np.load(pth, allow_pickle=False) for pth in paths)


def _save_cache(cache_dir, tag, arrays):
    os.makedirs(cache_dir, exist_ok=True)
    for nm, arr in zip(_NAMES, arrays):
        tmp = os.path.join(cache_dir, f"{tag}_{nm}.tmp.npy")
        np.save(tmp, arr, allow_pickle=False)
        os.replace(tmp, os.path.join(cache_dir, f"{tag}_{nm}.npy"))
