"""Every block length from 1 to 2 chunks and a bit, in both steps of the LDS
sweep (the folded one-column step and the general step) and in the sweep
with V in global memory, with one and with three passes per block: the last,
partial chunk of a block stops after the block's last rating, so each length
class (shorter than a chunk, exactly one or two chunks, a chunk plus a
remainder) must reproduce the oracle's epoch (Algorithm 1, Eq. 2-3) on the
same layout within the parity tolerance, and the two V placements must agree
bit for bit.

The layout: p = 8 row-blocks of 48 rows and 8 one-column column-blocks;
block (b, c) holds L(b, c) = 1 + (7b + 5c) mod 40 ratings on distinct rows
(no row repeats: the folded step), or, in the "repeats" variant, each block
with at least two ratings has its first row twice (the general step).
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
P, ROWS, K = 8, 48, 64


def _layout(repeats, seed=3):
    rng = np.random.default_rng(seed)
    rows, cols = [], []
    for b in range(P):
        for c in range(P):
            L = 1 + (7 * b + 5 * c) % 40
            r = b * ROWS + rng.choice(ROWS, size=L, replace=False)
            if repeats and L >= 2:
                r[1] = r[0]
            rows.append(r)
            cols.append(np.full(L, c))
    rows = np.concatenate(rows).astype(np.int32)
    cols = np.concatenate(cols).astype(np.int32)
    order = rng.permutation(len(rows))
    vals = rng.integers(1, 6, len(rows)).astype(np.float32)
    return rows[order], cols[order], vals[order]


def _gpu(rows, cols, vals, U0, V0, passes, v_staging, single=1):
    from paper_2304_13724_amd import bgmf
    n, m = P * ROWS, P
    with bgmf.Model(n, m, K, P) as mdl:
        mdl.set_cuts(np.arange(P + 1, dtype=np.int64) * ROWS, np.arange(P + 1, dtype=np.int64))
        mdl.set_option(bgmf.BGMF_OPT_BLOCK_PASSES, passes)
        mdl.set_option(bgmf.BGMF_OPT_V_STAGING, v_staging)
        mdl.set_option(bgmf.BGMF_OPT_SINGLE_COLUMN, single)
        mdl.set_factors(U0, V0)
        mdl.load_coo(rows, cols, vals)
        bp, perm = mdl.get_layout()
        for _ in range(2):
            mdl.epoch(0.02, 0.05)
        U, V = mdl.get_factors()
    return bp, perm, U, V


@pytest.mark.parametrize("repeats", [False, True], ids=["distinct_rows", "repeats"])
@pytest.mark.parametrize("passes", [1, 3])
def test_every_block_length(repeats, passes):
    rows, cols, vals = _layout(repeats)
    n, m = P * ROWS, P
    U0, V0 = init_factors(n, m, K, 11)
    print(f"block lengths: repeats={repeats} passes={passes} nnz={len(rows)}", flush=True)
    bp, perm, U, V = _gpu(rows, cols, vals, U0, V0, passes, v_staging=1)
    rc = np.arange(P + 1, dtype=np.int64) * ROWS
    cc = np.arange(P + 1, dtype=np.int64)
    obp, operm = oracle.bucket_cuts(n, m, P, rc, cc, rows, cols)
    assert np.array_equal(bp, obp) and np.array_equal(perm, operm)
    Uo, Vo = U0.copy(), V0.copy()
    for _ in range(2):
        oracle.epoch_passes(P, rows, cols, vals, obp, operm, Uo, Vo, 0.02, 0.05, passes, THREADS)
    assert row_rel_err(U, Uo) <= TOL and row_rel_err(V, Vo) <= TOL
    # V in global memory runs the general step: bit-identical to the LDS
    # sweep's general step
    _, _, Ug, Vg = _gpu(rows, cols, vals, U0, V0, passes, v_staging=2)
    _, _, Ul, Vl = _gpu(rows, cols, vals, U0, V0, passes, v_staging=1, single=0)
    assert np.array_equal(Ug, Ul) and np.array_equal(Vg, Vl)
    assert row_rel_err(Ul, Uo) <= TOL and row_rel_err(Vl, Vo) <= TOL
