"""Blocks of unequal size (bgmf_set_cuts): the HIP bucketing with given cut
points bit-exact against the oracle's, and the sweep against the oracle's
epoch on that layout, for balanced cut points (bgmf_balanced_cuts) and for
random ones, both V placements, streamed and in-core."""
import os

import numpy as np
import pytest

import oracle
from helpers import row_rel_err
from workloads import make, make_config

pytestmark = pytest.mark.gpu

TOL = 1e-4
THREADS = min(16, os.cpu_count() or 1)

CASES = {
    "medium_shape": lambda: make_config("medium", n=7_000, m=1_000, nnz=300_000, p=32),
    "large_shape": lambda: make_config("large", n=48_000, m=1_800, nnz=1_000_000, p=128),
    "k128_ragged": lambda: make("r", n=1_003, m=997, nnz=40_000, k=128, p=13, alpha=0.005,
                                beta=0.05, epochs=1, seed=61, structure="uniform",
                                values="int5", rank=4),
}


def _cuts(w, kind):
    from paper_2304_13724_amd import bgmf
    if kind == "balanced":
        cap = max(64, 2 * -(-w.m // w.p))  # narrow column-blocks, but enough to cover m
        return bgmf.bgmf_balanced_cuts(w.n, w.m, w.p, w.rows, w.cols, 65536, cap)
    rng = np.random.default_rng(w.p)
    rc = np.r_[0, np.sort(rng.choice(np.arange(1, w.n), w.p - 1, replace=False)), w.n]
    cc = np.r_[0, np.sort(rng.choice(np.arange(1, w.m), w.p - 1, replace=False)), w.m]
    return rc.astype(np.int64), cc.astype(np.int64)


def _gpu(w, rc, cc, epochs=1, v_staging=0, schedule=0, budget=0, single=1):
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_cuts(rc, cc)
        mdl.set_option(bgmf.BGMF_OPT_SINGLE_COLUMN, single)
        mdl.set_option(bgmf.BGMF_OPT_V_STAGING, v_staging)
        mdl.set_option(bgmf.BGMF_OPT_SCHEDULE, schedule)
        mdl.set_option(bgmf.BGMF_OPT_RATINGS_BUDGET, budget)
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        bp, perm = mdl.get_layout()
        hist = []
        for _ in range(epochs):
            mdl.epoch(w.alpha, w.beta)
            hist.append(mdl.rmse())
        U, V = mdl.get_factors()
        got = mdl.get_cuts()
    assert np.array_equal(got[0], rc) and np.array_equal(got[1], cc)
    return bp, perm, U, V, hist


def _oracle(w, rc, cc, epochs=1):
    bp, perm = oracle.bucket_cuts(w.n, w.m, w.p, rc, cc, w.rows, w.cols)
    U, V = w.U0.copy(), w.V0.copy()
    hist = []
    for _ in range(epochs):
        oracle.epoch_mt(w.p, w.rows, w.cols, w.vals, bp, perm, U, V, w.alpha, w.beta, THREADS)
        hist.append(oracle.rmse(w.rows, w.cols, w.vals, U, V))
    return bp, perm, U, V, hist


@pytest.mark.parametrize("case", sorted(CASES))
@pytest.mark.parametrize("kind", ["balanced", "random"])
def test_cuts_parity(case, kind):
    w = CASES[case]()
    rc, cc = _cuts(w, kind)
    g = _gpu(w, rc, cc, epochs=2)
    o = _oracle(w, rc, cc, epochs=2)
    assert np.array_equal(g[0], o[0]) and np.array_equal(g[1], o[1])
    assert row_rel_err(g[2], o[2]) <= TOL and row_rel_err(g[3], o[3]) <= TOL
    for a, b in zip(g[4], o[4]):
        assert abs(a - b) <= TOL * b


@pytest.mark.parametrize("v_staging,schedule", [(2, 0), (1, 1), (2, 2)])
def test_cuts_placements_bit_identical(v_staging, schedule):
    # V in global memory has no folded one-column step: compare it with the
    # general step of the LDS sweep (the folded step is checked against the
    # oracle above)
    single = 0 if v_staging == 2 else 1
    w = CASES["large_shape"]()
    rc, cc = _cuts(w, "balanced")
    a = _gpu(w, rc, cc, single=single)
    b = _gpu(w, rc, cc, v_staging=v_staging, schedule=schedule, single=single)
    assert np.array_equal(a[2], b[2]) and np.array_equal(a[3], b[3])


def test_cuts_streamed_bit_identical():
    w = CASES["large_shape"]()
    rc, cc = _cuts(w, "balanced")
    a = _gpu(w, rc, cc, epochs=2)
    b = _gpu(w, rc, cc, epochs=2, budget=w.nnz * 8 // 4)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert np.array_equal(a[2], b[2]) and np.array_equal(a[3], b[3])


def test_equal_cuts_are_the_default():
    from paper_2304_13724_amd import bgmf
    w = CASES["medium_shape"]()
    eq = lambda L: np.array([(R * L + w.p - 1) // w.p for R in range(w.p + 1)], dtype=np.int64)
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        rc, cc = mdl.get_cuts()
    assert np.array_equal(rc, eq(w.n)) and np.array_equal(cc, eq(w.m))
    a = _gpu(w, rc, cc)
    o = oracle.bucket(w.n, w.m, w.p, w.rows, w.cols)
    assert np.array_equal(a[0], o[0]) and np.array_equal(a[1], o[1])


def test_set_cuts_errors_and_reload():
    from paper_2304_13724_amd import bgmf
    w = CASES["medium_shape"]()
    rc, cc = _cuts(w, "balanced")
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        for bad_r, bad_c in [(rc[:-1], cc), (np.r_[rc[:-1], w.n + 1], cc),
                             (np.r_[0, rc[2:-1], rc[1], w.n], cc),
                             (rc, np.r_[0, 1, 1, cc[3:]])]:
            with pytest.raises((bgmf.BgmfError, ValueError)):
                if len(bad_r) != w.p + 1:
                    raise ValueError("wrong length")  # the ABI takes p + 1 values
                mdl.set_cuts(bad_r, bad_c)
        mdl.epoch(w.alpha, w.beta)  # the failed calls kept the loaded ratings
        mdl.set_cuts(rc, cc)
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.epoch(w.alpha, w.beta)  # new cuts drop the ratings
        assert ei.value.code == bgmf.BGMF_E_STATE
        mdl.load_coo(w.rows, w.cols, w.vals)
        mdl.epoch(w.alpha, w.beta)
        assert np.isfinite(mdl.rmse())
