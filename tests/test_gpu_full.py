"""GPU parity at the benchmark's full sizes, in the launch configuration
bench.py times (persistent schedule, default options).

* 100M ratings, k=64, p=1024: bucketing bit-exact against the oracle; U, V
  and RMSE after one epoch within 1e-4 of the oracle's multithreaded epoch
  (bit-identical to its sequential one).
* 10M ratings, k=32, p=256: three epochs, RMSE after each and final U, V.
"""
import os

import numpy as np
import pytest

import oracle
from helpers import row_rel_err
from workloads import make_config

pytestmark = [pytest.mark.gpu, pytest.mark.timeout(900)]

TOL = 1e-4
THREADS = min(16, os.cpu_count() or 1)
CACHE = os.environ.get("BGMF_WORKLOAD_CACHE", "/tmp/bgmf_cache")


def _gpu(w, epochs):
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        bp, perm = mdl.get_layout()
        hist = []
        for _ in range(epochs):
            mdl.epoch(w.alpha, w.beta)
            hist.append(mdl.rmse())
        U, V = mdl.get_factors()
    return bp, perm, U, V, hist


def _oracle(w, epochs):
    bp, perm = oracle.bucket(w.n, w.m, w.p, w.rows, w.cols)
    U, V = w.U0.copy(), w.V0.copy()
    hist = []
    for _ in range(epochs):
        oracle.epoch_mt(w.p, w.rows, w.cols, w.vals, bp, perm, U, V, w.alpha, w.beta, THREADS)
        hist.append(oracle.rmse(w.rows, w.cols, w.vals, U, V))
    return bp, perm, U, V, hist


@pytest.fixture(scope="module")
def large():
    w = make_config("large", cache_dir=CACHE)
    print(f"large workload: nnz={w.nnz}", flush=True)
    return w, _gpu(w, 1), _oracle(w, 1)


def test_large_bucketing_bit_exact(large):
    w, g, o = large
    assert np.array_equal(g[0], o[0])
    assert np.array_equal(g[1], o[1])


def test_large_one_epoch_parity(large):
    w, g, o = large
    assert row_rel_err(g[2], o[2]) <= TOL
    assert row_rel_err(g[3], o[3]) <= TOL
    assert abs(g[4][0] - o[4][0]) <= TOL * o[4][0]


def test_medium_three_epochs():
    w = make_config("medium", cache_dir=CACHE)
    g = _gpu(w, 3)
    o = _oracle(w, 3)
    assert np.array_equal(g[0], o[0]) and np.array_equal(g[1], o[1])
    for a, b in zip(g[4], o[4]):
        assert abs(a - b) <= TOL * b
    assert row_rel_err(g[2], o[2]) <= 3 * TOL
    assert row_rel_err(g[3], o[3]) <= 3 * TOL
