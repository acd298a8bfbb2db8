"""Seeded random configurations through the C ABI against the oracle: shape
(n, m, nnz including duplicate ratings and empty rows), k (padded widths
too), p (from 1), equal or random cut points, block passes, schedule, V
placement, and a ratings budget that makes them stream.  Each case: the
layout bit-exact against the oracle's bucketing, U and V after each of two
epochs within 1e-4 (row-normwise), and the RMSE within 1e-4 relative.

The inputs are drawn here from a seeded generator (no method arithmetic);
the draw of each case is printed so a failure names it.
"""
import os

import numpy as np
import pytest

import oracle
from helpers import row_rel_err
from workloads import init_factors

pytestmark = pytest.mark.gpu

TOL = 1e-4
THREADS = min(16, os.cpu_count() or 1)
CASES = 64


def _draw(seed):
    rng = np.random.default_rng(1000 + seed)
    n = int(rng.integers(1, 4000))
    m = int(rng.integers(1, 2500))
    p = int(rng.integers(1, min(n, m, 48) + 1))
    k = int(rng.choice([16, 32, 48, 64, 80, 128, 256]))
    nnz = int(rng.integers(1, 40_000))
    rows = rng.integers(0, n, nnz).astype(np.int32)
    cols = rng.integers(0, m, nnz).astype(np.int32)
    if nnz > 10 and rng.random() < 0.5:  # repeat some (row, column) pairs
        d = rng.integers(0, nnz, nnz // 10)
        rows[d[: len(d) // 2]] = rows[d[len(d) // 2: 2 * (len(d) // 2)]]
        cols[d[: len(d) // 2]] = cols[d[len(d) // 2: 2 * (len(d) // 2)]]
    vals = rng.integers(1, 6, nnz).astype(np.float32)
    U0, V0 = init_factors(n, m, k, 2000 + seed)
    cuts = None
    if rng.random() < 0.4 and p > 1:
        rc = np.r_[0, np.sort(rng.choice(np.arange(1, n), p - 1, replace=False)), n]
        cc = np.r_[0, np.sort(rng.choice(np.arange(1, m), p - 1, replace=False)), m]
        if np.diff(cc).max() <= 65536:
            cuts = (rc.astype(np.int64), cc.astype(np.int64))
    opts = dict(
        passes=int(rng.choice([1, 1, 2])),
        schedule=int(rng.choice([0, 1, 2])),
        v_staging=int(rng.choice([0, 2])),
        stream=bool(rng.random() < 0.3 and p > 1),
    )
    alpha = float(rng.choice([0.005, 0.01, 0.02]))
    beta = float(rng.choice([0.0, 0.05]))
    return dict(n=n, m=m, k=k, p=p, rows=rows, cols=cols, vals=vals, U0=U0, V0=V0, cuts=cuts,
                alpha=alpha, beta=beta, **opts)


def _gpu(c, epochs):
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(c["n"], c["m"], c["k"], c["p"]) as mdl:
        if c["cuts"] is not None:
            mdl.set_cuts(*c["cuts"])
        mdl.set_option(bgmf.BGMF_OPT_BLOCK_PASSES, c["passes"])
        mdl.set_option(bgmf.BGMF_OPT_SCHEDULE, c["schedule"])
        mdl.set_option(bgmf.BGMF_OPT_V_STAGING, c["v_staging"])
        if c["stream"]:
            # about half of the records on the device, the rest streamed
            mdl.set_option(bgmf.BGMF_OPT_RATINGS_BUDGET, max(len(c["rows"]) * 8 // 2, 1 << 16))
        mdl.set_factors(c["U0"], c["V0"])
        mdl.load_coo(c["rows"], c["cols"], c["vals"])
        bp, perm = mdl.get_layout()
        hist = []
        for _ in range(epochs):
            mdl.epoch(c["alpha"], c["beta"])
            hist.append((mdl.rmse(),) + mdl.get_factors())
    return bp, perm, hist


def _oracle(c, epochs):
    if c["cuts"] is None:
        bp, perm = oracle.bucket(c["n"], c["m"], c["p"], c["rows"], c["cols"])
    else:
        bp, perm = oracle.bucket_cuts(c["n"], c["m"], c["p"], c["cuts"][0], c["cuts"][1],
                                      c["rows"], c["cols"])
    U, V = c["U0"].copy(), c["V0"].copy()
    hist = []
    for _ in range(epochs):
        oracle.epoch_passes(c["p"], c["rows"], c["cols"], c["vals"], bp, perm, U, V, c["alpha"],
                            c["beta"], c["passes"], THREADS)
        hist.append((oracle.rmse(c["rows"], c["cols"], c["vals"], U, V), U.copy(), V.copy()))
    return bp, perm, hist


@pytest.mark.parametrize("seed", range(CASES))
def test_random_configuration(seed):
    c = _draw(seed)
    print(f"case {seed}: n={c['n']} m={c['m']} k={c['k']} p={c['p']} nnz={len(c['rows'])} "
          f"cuts={'random' if c['cuts'] is not None else 'equal'} passes={c['passes']} "
          f"schedule={c['schedule']} v_staging={c['v_staging']} stream={c['stream']} "
          f"alpha={c['alpha']} beta={c['beta']}", flush=True)
    g_bp, g_perm, g = _gpu(c, 2)
    o_bp, o_perm, o = _oracle(c, 2)
    assert np.array_equal(g_bp, o_bp) and np.array_equal(g_perm, o_perm)
    for (gr, gU, gV), (orr, oU, oV) in zip(g, o):
        assert row_rel_err(gU, oU) <= TOL and row_rel_err(gV, oV) <= TOL
        assert abs(gr - orr) <= TOL * max(orr, 1e-12)
