"""The library's nnz-balanced cut points (bgmf_balanced_cuts), a host-only
function: checked without a GPU against an independent numpy statement of
its rule and against the invariants every cut table must meet."""
import numpy as np
import pytest

from workloads import make, make_config


def _rule(deg, p, cap):
    """Block b ends at the first index where the running count reaches
    ceil(remaining / blocks left), or just before it if that index alone
    holds the share; kept within [prev + 1, prev + cap], leaving each later
    block at least one index and at most cap."""
    cum = np.concatenate([[0], np.cumsum(deg)]).astype(np.int64)
    L = len(deg)
    total = int(cum[-1])
    cut = [0]
    for b in range(1, p):
        prev = cut[-1]
        left = p - b + 1
        target = int(cum[prev]) + -(-(total - int(cum[prev])) // left)
        c = prev + 1 + int(np.searchsorted(cum[prev + 1:], target, side="left"))
        if c <= L and c - 1 > prev and deg[c - 1] >= target - int(cum[prev]):
            c -= 1  # a heavy index starts its own block
        c = max(c, prev + 1)
        c = min(c, prev + cap, L - (p - b))
        c = max(c, L - (p - b) * cap)
        cut.append(c)
    cut.append(L)
    return np.array(cut, dtype=np.int64)


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
    rd = np.bincount(w.rows, minlength=w.n)
    cd = np.bincount(w.cols, minlength=w.m)
    assert np.array_equal(rc, _rule(rd, w.p, min(cap_rows, 65536)))
    assert np.array_equal(cc, _rule(cd, w.p, min(cap_cols, 16384)))
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
