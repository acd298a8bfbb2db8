"""The library's degree-aware relabelling (bgmf_reorder_ids), a host-only
function: checked without a GPU against the optimum found by exhaustive
search on tiny inputs and against the properties its statement fixes."""
import itertools

import numpy as np
import pytest

from workloads import make_config


def _equal_cuts(length, p):
    return [-(-b * length // p) for b in range(p + 1)]


def _best_max_load(deg, p):
    """Smallest possible largest block load over every placement of the
    indices into the paper's p equal-width blocks (brute force)."""
    cut = _equal_cuts(len(deg), p)
    labels = [b for b in range(p) for _ in range(cut[b + 1] - cut[b])]
    best = None
    for perm in set(itertools.permutations(labels)):
        loads = [0] * p
        for i, b in enumerate(perm):
            loads[b] += int(deg[i])
        best = max(loads) if best is None else min(best, max(loads))
    return best


def test_relabelling_against_exhaustive_search():
    """300 random degree vectors (2..7 indices, a heavy index in a third of
    them) over 1..3 blocks: the new ids are a permutation, the heaviest index
    (lowest id among ties) gets id 0 (it is dealt first, to block 0), and the
    largest block load is within 1.5 times the best possible (the deal is
    longest-processing-time-first; 1.5 is the worst ratio it reached on
    these inputs)."""
    from paper_2304_13724_amd import bgmf
    rng = np.random.default_rng(13724)
    for _ in range(300):
        L = int(rng.integers(2, 8))
        p = int(rng.integers(1, min(L, 3) + 1))
        deg = rng.integers(0, 8, L)
        if rng.random() < 0.3:
            deg[rng.integers(0, L)] += int(rng.integers(5, 30))
        if deg.sum() == 0:
            deg[0] = 1
        rows = np.repeat(np.arange(L), deg).astype(np.int32)
        rn, cn = bgmf.bgmf_reorder_ids(L, L, p, rows, np.zeros_like(rows))
        assert sorted(rn.tolist()) == list(range(L))
        assert rn[int(np.argmax(deg))] == 0
        new_deg = np.zeros(L, dtype=np.int64)
        new_deg[rn] = deg
        cut = _equal_cuts(L, p)
        loads = [int(new_deg[cut[b]:cut[b + 1]].sum()) for b in range(p)]
        assert 2 * max(loads) <= 3 * _best_max_load(deg, p), (deg.tolist(), p, rn.tolist())


@pytest.mark.parametrize("shape", ["medium", "large"])
def test_relabelling_spreads_heavy_items(shape):
    """On workload-shaped inputs: both relabellings are permutations, and
    every block's load is at most the mean load plus the heaviest single
    index (an index cannot be split), for rows and for columns."""
    from paper_2304_13724_amd import bgmf
    w = (make_config("medium", n=7_000, m=1_000, nnz=300_000, p=32) if shape == "medium"
         else make_config("large", n=48_000, m=1_800, nnz=1_000_000, p=128))
    rn, cn = bgmf.bgmf_reorder_ids(w.n, w.m, w.p, w.rows, w.cols)
    for newid, idx, length in ((rn, w.rows, w.n), (cn, w.cols, w.m)):
        assert np.array_equal(np.sort(newid), np.arange(length))
        deg = np.bincount(idx, minlength=length)
        new_deg = np.zeros(length, dtype=np.int64)
        new_deg[newid] = deg
        loads = np.add.reduceat(new_deg, np.array(_equal_cuts(length, w.p)[:-1]))
        assert loads.max() <= w.nnz / w.p + deg.max()


def test_relabelling_errors():
    from paper_2304_13724_amd import bgmf
    rows = np.array([0, 1, 2], dtype=np.int32)
    cols = np.array([0, 1, 2], dtype=np.int32)
    with pytest.raises(bgmf.BgmfError) as ei:
        bgmf.bgmf_reorder_ids(3, 3, 4, rows, cols)  # p > n
    assert ei.value.code == bgmf.BGMF_E_ARG
    with pytest.raises(bgmf.BgmfError) as ei:
        bgmf.bgmf_reorder_ids(3, 3, 1, rows, np.array([0, 1, 3], dtype=np.int32))
    assert ei.value.code == bgmf.BGMF_E_RANGE
