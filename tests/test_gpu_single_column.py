"""Blocks of a one-column column-block (BGMF_OPT_SINGLE_COLUMN).  A block in
which no row repeats in consecutive ratings takes the folded step (v in
registers for the whole block, the next rating's partial products formed
before e is known): the stored u and v are updated as in the general step,
only the rounding of the next dot product differs, so it must match the
oracle's epoch (Algorithm 1, Eq. 2-3) on the same layout within the parity
tolerance.  A block that repeats a row (a duplicate rating) takes the
general step, so with every one-column block holding a duplicate the option
changes no bit.

The crafted workload puts one heavy column alone in each of the first three
column-blocks (every user rates it) and plants duplicates: one whose two
copies straddle a chunk boundary, one inside a chunk, in some row-blocks
only (those blocks take the general step, the others fold), blocks whose
length is not a multiple of the chunk, and a column-block with many columns
beside them.
"""
import os

import numpy as np
import pytest

import oracle
from helpers import row_rel_err
from workloads import init_factors, make_config

pytestmark = pytest.mark.gpu

TOL = 1e-4
THREADS = min(16, os.cpu_count() or 1)


class _W:
    pass


def _crafted(k, seed=7, dup_all=False):
    """n users, heavy columns 0, 1, 2 in column-blocks of their own, the other
    columns in the last block; duplicates of rows 15 (copies at block
    positions 15 and 16) and 40 in every heavy column, and of row 520 of
    column 1 (second row-block).  ``dup_all``: also a duplicate in every
    row-block of every heavy column."""
    n, m, p = 2_000, 61, 4
    rng = np.random.default_rng(seed)
    rows, cols = [], []
    for j in (0, 1, 2):
        r = np.arange(n)
        r = np.sort(np.r_[r, 15, 40, 520 if j == 1 else 41])
        if dup_all:
            r = np.sort(np.r_[r, 600, 1100, 1700])
        rows.append(r)
        cols.append(np.full(len(r), j))
    extra = 30_000
    rows.append(rng.integers(0, n, extra))
    cols.append(rng.integers(3, m, extra))
    rows = np.concatenate(rows).astype(np.int32)
    cols = np.concatenate(cols).astype(np.int32)
    order = rng.permutation(len(rows))  # input order does not matter to the layout
    w = _W()
    w.n, w.m, w.k, w.p = n, m, k, p
    w.rows, w.cols = rows[order], cols[order]
    w.vals = rng.integers(1, 6, len(rows)).astype(np.float32)
    w.U0, w.V0 = init_factors(n, m, k, seed)
    w.alpha, w.beta = 0.01, 0.05
    rc = np.array([(R * n + p - 1) // p for R in range(p + 1)], dtype=np.int64)
    cc = np.array([0, 1, 2, 3, m], dtype=np.int64)
    return w, rc, cc


def _gpu(w, rc, cc, single, epochs=2, schedule=0, passes=1):
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_cuts(rc, cc)
        mdl.set_option(bgmf.BGMF_OPT_V_STAGING, 1)
        mdl.set_option(bgmf.BGMF_OPT_SCHEDULE, schedule)
        mdl.set_option(bgmf.BGMF_OPT_BLOCK_PASSES, passes)
        mdl.set_option(bgmf.BGMF_OPT_SINGLE_COLUMN, single)
        assert mdl.get_option(bgmf.BGMF_OPT_SINGLE_COLUMN) == single
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        hist = []
        for _ in range(epochs):
            mdl.epoch(w.alpha, w.beta)
            hist.append(mdl.rmse())
        U, V = mdl.get_factors()
    return U, V, hist


def _oracle(w, rc, cc, epochs=2, passes=1):
    bp, perm = oracle.bucket_cuts(w.n, w.m, w.p, rc, cc, w.rows, w.cols)
    U, V = w.U0.copy(), w.V0.copy()
    hist = []
    for _ in range(epochs):
        if passes == 1:
            oracle.epoch_mt(w.p, w.rows, w.cols, w.vals, bp, perm, U, V, w.alpha, w.beta,
                            THREADS)
        else:
            oracle.epoch_passes(w.p, w.rows, w.cols, w.vals, bp, perm, U, V, w.alpha, w.beta,
                                passes)
        hist.append(oracle.rmse(w.rows, w.cols, w.vals, U, V))
    return U, V, hist


def test_crafted_layout_has_the_planted_cases():
    w, rc, cc = _crafted(64)
    bp, perm = oracle.bucket_cuts(w.n, w.m, w.p, rc, cc, w.rows, w.cols)
    p = w.p
    # block (R = 0, C = 0) is stratum 0, slot 0: positions 15 and 16 hold row 15
    blk = perm[bp[0]:bp[1]]
    assert np.all(w.cols[blk] == 0)
    assert w.rows[blk][15] == 15 and w.rows[blk][16] == 15
    # block (R = 1, C = 1) is stratum 0, slot 1: holds the duplicate of row 520
    blk = perm[bp[1]:bp[2]]
    r = w.rows[blk]
    assert np.all(w.cols[blk] == 1) and np.count_nonzero(r == 520) == 2
    assert bp[p * p] == len(w.rows)
    # one-column blocks whose length is not a multiple of 16
    sizes = np.diff(bp).reshape(p, p)  # [s, R]; column-block (R + s) mod p
    one = [sizes[s, R] for s in range(p) for R in range(p) if (R + s) % p < 3]
    assert any(x % 16 for x in one)


def _check_oracle(g, o):
    assert row_rel_err(g[0], o[0]) <= TOL and row_rel_err(g[1], o[1]) <= TOL
    for a, b in zip(g[2], o[2]):
        assert abs(a - b) <= TOL * b


@pytest.mark.parametrize("k", [16, 48, 64, 128])
@pytest.mark.parametrize("schedule", [0, 1])
def test_crafted_fold_and_oracle(k, schedule):
    w, rc, cc = _crafted(k)
    o = _oracle(w, rc, cc)
    _check_oracle(_gpu(w, rc, cc, 1, schedule=schedule), o)
    _check_oracle(_gpu(w, rc, cc, 0, schedule=schedule), o)


@pytest.mark.parametrize("k", [16, 64, 128])
def test_repeated_rows_take_the_general_step(k):
    w, rc, cc = _crafted(k, dup_all=True)
    on = _gpu(w, rc, cc, 1)
    off = _gpu(w, rc, cc, 0)
    assert np.array_equal(on[0], off[0]) and np.array_equal(on[1], off[1])
    assert on[2] == off[2]
    _check_oracle(on, _oracle(w, rc, cc))


def test_crafted_passes():
    w, rc, cc = _crafted(64)
    o = _oracle(w, rc, cc, epochs=1, passes=3)
    for single in (1, 0):
        g = _gpu(w, rc, cc, single, epochs=1, passes=3)
        assert row_rel_err(g[0], o[0]) <= TOL and row_rel_err(g[1], o[1]) <= TOL


def test_balanced_heavy_items_oracle():
    """Zipf items with nnz-balanced cut points (heavy items isolated, their
    blocks take the folded step), two epochs against the oracle."""
    from paper_2304_13724_amd import bgmf
    w = make_config("large", n=48_000, m=1_800, nnz=1_000_000, p=128)
    rc, cc = bgmf.bgmf_balanced_cuts(w.n, w.m, w.p, w.rows, w.cols, 65536, 64)
    assert int(np.diff(cc).min()) == 1  # some column-blocks hold one item
    _check_oracle(_gpu(w, rc, cc, 1), _oracle(w, rc, cc))


def test_fold_correction_term_is_exercised():
    """One column rated by every user, factors drawn wide and a large step,
    so that the term carried by the folded step (e times a u'.u) is several
    percent of the next error: a wrong or missing term would miss the
    oracle by far more than the tolerance."""
    n, m, k, p = 3_000, 8, 64, 4
    rng = np.random.default_rng(31)
    rows = np.r_[np.arange(n), rng.integers(0, n, 4_000)].astype(np.int32)
    cols = np.r_[np.zeros(n, np.int64), rng.integers(1, m, 4_000)].astype(np.int32)
    order = rng.permutation(len(rows))
    w = _W()
    w.n, w.m, w.k, w.p = n, m, k, p
    w.rows, w.cols = rows[order], cols[order]
    w.vals = rng.integers(1, 6, len(rows)).astype(np.float32)
    w.U0 = rng.normal(0.0, 0.3, (n, k)).astype(np.float32)
    w.V0 = rng.normal(0.0, 0.3, (m, k)).astype(np.float32)
    w.alpha, w.beta = 0.05, 0.05
    rc = np.array([(R * n + p - 1) // p for R in range(p + 1)], dtype=np.int64)
    cc = np.array([0, 1, 2, 3, m], dtype=np.int64)
    # size of the folded term along the first block of column 0 (rows in
    # ascending order), in binary64 with the plain update
    U = w.U0.astype(np.float64)
    v = w.V0[0].astype(np.float64)
    x = np.zeros(n)
    x[rows[:n]] = w.vals[np.argsort(order)][:n]
    ratio = 0.0
    for i in range(rc[1] - 1):
        e = x[i] - U[i] @ v
        u = U[i].copy()
        U[i] += w.alpha * (e * v - w.beta * U[i])
        v += w.alpha * (e * u - w.beta * v)
        ratio = max(ratio, abs(e * w.alpha * (U[i + 1] @ u)) / (abs(x[i + 1] - U[i + 1] @ v) + 1e-3))
    assert ratio > 0.05
    o = _oracle(w, rc, cc)
    _check_oracle(_gpu(w, rc, cc, 1), o)


def test_one_distinct_column_in_wider_blocks():
    """The paper's equal blocks (16 columns wide), where every block of
    column-block 0 has all its ratings on column 5 (each user rates it once)
    and the other column-blocks are ordinary: those blocks take the folded
    step although their column-block is wider than one column (the option
    then changes the last bits of column 5, which shows the fold ran), and one epoch
    matches the oracle within the tolerance either way."""
    from paper_2304_13724_amd import bgmf
    n, m, p, k = 2_000, 64, 4, 64
    rng = np.random.default_rng(23)
    rows = np.r_[np.arange(n), rng.integers(0, n, 20_000)].astype(np.int32)
    cols = np.r_[np.full(n, 5), rng.integers(16, m, 20_000)].astype(np.int32)
    order = rng.permutation(len(rows))
    w = _W()
    w.n, w.m, w.k, w.p = n, m, k, p
    w.rows, w.cols = rows[order], cols[order]
    w.vals = rng.integers(1, 6, len(rows)).astype(np.float32)
    w.U0, w.V0 = init_factors(n, m, k, 3)
    w.alpha, w.beta = 0.01, 0.05
    bp, perm = oracle.bucket(n, m, p, w.rows, w.cols)
    Uo, Vo = w.U0.copy(), w.V0.copy()
    oracle.epoch(p, w.rows, w.cols, w.vals, bp, perm, Uo, Vo, w.alpha, w.beta)
    out = {}
    for single in (1, 0):
        with bgmf.Model(n, m, k, p) as mdl:
            mdl.set_option(bgmf.BGMF_OPT_SINGLE_COLUMN, single)
            mdl.set_factors(w.U0, w.V0)
            mdl.load_coo(w.rows, w.cols, w.vals)
            assert mdl.get_option(bgmf.BGMF_OPT_PLACEMENT) & 1  # V staged in LDS
            mdl.epoch(w.alpha, w.beta)
            out[single] = mdl.get_factors()
        du, dv = row_rel_err(out[single][0], Uo), row_rel_err(out[single][1], Vo)
        print(f"single_column={single}: row rel err U {du:.3e} V {dv:.3e}", flush=True)
        assert du <= TOL and dv <= TOL
    assert not np.array_equal(out[1][1][5], out[0][1][5])  # column 5 went through the fold
