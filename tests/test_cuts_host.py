"""The library's nnz-balanced cut points (bgmf_balanced_cuts), a host-only
function: checked without a GPU against the optimum found by exhaustive
search on tiny inputs (the largest block load stays within twice the best
possible over all contiguous cuttings), and against the invariants every cut
table must meet on workload-shaped inputs."""
import itertools

import numpy as np
import pytest

from workloads import make, make_config


def _best_max_load(deg, p):
    """Smallest possible largest block load over every way to cut the
    indices 0..L-1 into p non-empty contiguous blocks (brute force)."""
    L = len(deg)
    best = None
    for cuts in itertools.combinations(range(1, L), p - 1):
        c = (0, *cuts, L)
        mx = max(int(deg[c[i]:c[i + 1]].sum()) for i in range(p))
        best = mx if best is None else min(best, mx)
    return best


def test_balanced_cuts_within_twice_the_optimum():
    """800 random degree vectors of 2..10 indices (zeros, and a heavy index
    in a third of them) cut into 1..5 blocks: the library's largest block
    load is at most twice the exhaustive-search optimum, and every block is
    non-empty."""
    from paper_2304_13724_amd import bgmf
    rng = np.random.default_rng(2304)
    for _ in range(800):
        L = int(rng.integers(2, 11))
        p = int(rng.integers(1, min(L, 5) + 1))
        deg = rng.integers(0, 6, L) * (rng.random(L) < 0.8)
        if rng.random() < 0.3:
            deg[rng.integers(0, L)] += int(rng.integers(5, 40))
        if deg.sum() == 0:
            deg[0] = 1
        rows = np.repeat(np.arange(L), deg).astype(np.int32)
        rc, _ = bgmf.bgmf_balanced_cuts(L, L, p, rows, np.zeros_like(rows), 65536, 65536)
        assert rc[0] == 0 and rc[-1] == L and np.all(np.diff(rc) >= 1)
        loads = np.add.reduceat(deg, rc[:-1])
        assert loads.max() <= 2 * _best_max_load(deg, p), (deg.tolist(), p, rc.tolist())


@pytest.mark.parametrize("case,cap_rows,cap_cols", [
    ("medium_shape", 65536, 16384),
    ("medium_shape", 400, 60),
    ("large_shape", 65536, 40),
    ("uniform", 65536, 16384),
])
def test_balanced_cuts(case, cap_rows, cap_cols):
    from paper_2304_13724_amd import bgmf
    if case == "medium_shape":
        w = make_config("medium", n=7_000, m=1_000, nnz=300_000, p=32)
    elif case == "large_shape":
        w = make_config("large", n=48_000, m=1_800, nnz=1_000_000, p=128)
    else:
        w = make("u", n=2_000, m=900, nnz=50_000, k=16, p=16, alpha=0.01, beta=0.05, epochs=1,
                 seed=51, structure="uniform", values="int5", rank=4)
    rc, cc = bgmf.bgmf_balanced_cuts(w.n, w.m, w.p, w.rows, w.cols, cap_rows, cap_cols)
    cd = np.bincount(w.cols, minlength=w.m)
    for cut, length, cap in ((rc, w.n, cap_rows), (cc, w.m, cap_cols)):
        assert cut[0] == 0 and cut[-1] == length and len(cut) == w.p + 1
        widths = np.diff(cut)
        assert widths.min() >= 1 and widths.max() <= cap
    # balance: no column-block holds more than twice the mean plus its
    # heaviest single column (one column cannot be split)
    per = np.add.reduceat(cd, cc[:-1])
    assert per.max() <= 2 * w.nnz / w.p + cd.max()


def test_balanced_cuts_errors():
    from paper_2304_13724_amd import bgmf
    rows = np.array([0, 1, 2], dtype=np.int32)
    cols = np.array([0, 1, 2], dtype=np.int32)
    with pytest.raises(bgmf.BgmfError) as ei:
        bgmf.bgmf_balanced_cuts(3, 3, 4, rows, cols)          # p > n
    assert ei.value.code == bgmf.BGMF_E_ARG
    with pytest.raises(bgmf.BgmfError) as ei:
        bgmf.bgmf_balanced_cuts(100, 3, 2, rows, cols, 10, 2)  # 2 blocks of <= 10 rows < 100
    assert ei.value.code == bgmf.BGMF_E_ARG
    with pytest.raises(bgmf.BgmfError) as ei:
        bgmf.bgmf_balanced_cuts(3, 3, 1, rows, np.array([0, 1, 3], dtype=np.int32))
    assert ei.value.code == bgmf.BGMF_E_RANGE
