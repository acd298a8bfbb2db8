"""Sweep with V in global memory (no LDS staging of the column slice).

That variant prefetches every v row ahead of use and patches the prefetch
with the results of the recent ratings of the same column, so its
arithmetic is the same as the LDS-staged sweep, step for step: results must
be bit-identical to it, and match the oracle.  The cases stress the patch
logic (columns repeating at every distance inside a block) and the shapes
whose column slice does not fit in LDS at all.
"""
import numpy as np
import pytest

from helpers import gpu_run, oracle_run, row_rel_err
from workloads import make, make_config

pytestmark = pytest.mark.gpu

TOL = 1e-4
LDS, GLOBAL = 1, 2


def _dup(n, m, nnz, k, p, seed, hot=None):
    """Uniform ratings with repeated (i, j) pairs allowed; ``hot`` > 0 draws
    columns from a geometric law, so a few columns of each block repeat at
    short distances."""
    from workloads.synth import Workload, init_factors
    rng = np.random.default_rng(seed)
    rows = rng.integers(0, n, nnz).astype(np.int32)
    if hot:
        cols = np.minimum(rng.geometric(hot, nnz) - 1, m - 1).astype(np.int32)
    else:
        cols = rng.integers(0, m, nnz).astype(np.int32)
    vals = rng.integers(1, 6, nnz).astype(np.float32)
    U0, V0 = init_factors(n, m, k, seed + 100)
    return Workload("dup", n, m, k, p, 0.01, 0.05, 1, rows, cols, vals, U0, V0)


CASES = {
    "tiny": lambda: make_config("tiny"),
    "medium_shape": lambda: make_config("medium", n=7_000, m=1_000, nnz=300_000, p=32),
    "large_shape": lambda: make_config("large", n=48_000, m=1_800, nnz=1_000_000, p=128),
    # 16 columns per block, ~6,700 ratings per block: every repeat distance
    "hot_16cols": lambda: _dup(3_000, 48, 60_000, 64, 3, 21),
    # one column carries most ratings: long runs of distance 1
    "hot_geometric": lambda: _dup(2_000, 400, 50_000, 32, 4, 22, hot=0.3),
    "p1": lambda: _dup(300, 200, 5_000, 16, 1, 23),
    "ragged_k80": lambda: make("r", n=1_003, m=997, nnz=40_000, k=80, p=13, alpha=0.01,
                               beta=0.05, epochs=1, seed=24, structure="uniform",
                               values="int5", rank=4),
    "k256": lambda: make("w", n=2_000, m=900, nnz=50_000, k=256, p=8, alpha=0.005,
                         beta=0.05, epochs=1, seed=25, structure="uniform", values="int5",
                         rank=4),
}


@pytest.mark.parametrize("case", sorted(CASES))
@pytest.mark.parametrize("schedule", [0, 1, 2])
def test_bit_identical_to_lds(case, schedule):
    w = CASES[case]()
    a = gpu_run(w, 2, schedule=schedule, v_staging=LDS, single=0)
    g = gpu_run(w, 2, schedule=schedule, v_staging=GLOBAL)
    assert np.array_equal(g[0], a[0]) and np.array_equal(g[1], a[1])
    assert g[2] == a[2]


@pytest.mark.parametrize("case", ["hot_16cols", "hot_geometric", "ragged_k80", "k256"])
def test_oracle_parity(case):
    w = CASES[case]()
    U_ref, V_ref, hist_ref, _, _ = oracle_run(w, 2)
    U, V, hist, _, _ = gpu_run(w, 2, v_staging=GLOBAL)
    assert row_rel_err(U, U_ref) <= TOL and row_rel_err(V, V_ref) <= TOL
    for x, y in zip(hist, hist_ref):
        assert abs(x - y) <= TOL * y


def _cycle(d, k, reps=40, p=1):
    """One rating per row, rows ascending, columns cycling through d values:
    inside a block every column comes back after exactly d ratings (d = 1:
    one column throughout).  With p = 1 the whole matrix is one block."""
    from workloads.synth import Workload, init_factors
    n = d * reps + 3
    rows = np.arange(n, dtype=np.int32)
    cols = (rows % d).astype(np.int32)
    vals = (1 + rows % 5).astype(np.float32)
    U0, V0 = init_factors(n, max(d, 2), k, 300 + d)
    return Workload("cycle", n, max(d, 2), k, p, 0.01, 0.05, 1, rows, cols, vals, U0, V0)


@pytest.mark.parametrize("k", [64, 128])
@pytest.mark.parametrize("d", [1, 2, 3, 13, 14, 15, 16, 17, 31])
def test_repeat_distance(d, k):
    """A column repeated at exactly distance d.  A rating's v row is
    prefetched 16 ratings ahead, so it misses the updates of the ratings in
    between: at k = 128 those at distance 1..15 (a rating's store precedes
    the prefetch issued in its step), at k <= 64 those at 1..16 (the store
    is deferred into the next step).  The latest result must replace the
    prefetch there, and the prefetch is used as loaded beyond: d = 15, 16
    and 17 are the edges."""
    w = _cycle(d, k)
    a = gpu_run(w, 2, v_staging=LDS, single=0)
    g = gpu_run(w, 2, v_staging=GLOBAL)
    assert np.array_equal(g[0], a[0]) and np.array_equal(g[1], a[1])
    U_ref, V_ref, hist_ref, _, _ = oracle_run(w, 2)
    assert row_rel_err(g[0], U_ref) <= TOL and row_rel_err(g[1], V_ref) <= TOL
    for x, y in zip(g[2], hist_ref):
        assert abs(x - y) <= TOL * y


def test_placement_option():
    from paper_2304_13724_amd import bgmf
    w = CASES["medium_shape"]()
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        assert mdl.get_option(bgmf.BGMF_OPT_PLACEMENT) == 1 | 4  # fits: LDS, persistent
        mdl.set_option(bgmf.BGMF_OPT_V_STAGING, GLOBAL)
        assert mdl.get_option(bgmf.BGMF_OPT_PLACEMENT) == 2  # automatic: per stratum
        mdl.set_option(bgmf.BGMF_OPT_SCHEDULE, 2)
        assert mdl.get_option(bgmf.BGMF_OPT_PLACEMENT) == 2 | 4
        mdl.set_option(bgmf.BGMF_OPT_SCHEDULE, 1)
        assert mdl.get_option(bgmf.BGMF_OPT_PLACEMENT) == 2
        mdl.set_option(bgmf.BGMF_OPT_V_STAGING, LDS)
        assert mdl.get_option(bgmf.BGMF_OPT_PLACEMENT) == 1
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.set_option(bgmf.BGMF_OPT_V_STAGING, 3)
        assert ei.value.code == bgmf.BGMF_E_ARG


@pytest.mark.parametrize("schedule", [0, 1, 2])
def test_slice_wider_than_lds(schedule):
    """k=256 and 469 columns per block: a slice needs 470 KiB, more than a
    workgroup's LDS, so only the global-memory sweep can run it."""
    from paper_2304_13724_amd import bgmf
    w = make("wide", n=3_000, m=60_000, nnz=150_000, k=256, p=128, alpha=0.005, beta=0.05,
             epochs=1, seed=26, structure="uniform", values="int5", rank=4)
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.set_option(bgmf.BGMF_OPT_V_STAGING, LDS)
        assert ei.value.code == bgmf.BGMF_E_UNSUPPORTED
        mdl.set_option(bgmf.BGMF_OPT_SCHEDULE, schedule)
        assert mdl.get_option(bgmf.BGMF_OPT_PLACEMENT) & 2
    U_ref, V_ref, hist_ref, _, _ = oracle_run(w, 2)
    U, V, hist, _, _ = gpu_run(w, 2, schedule=schedule)
    assert row_rel_err(U, U_ref) <= TOL and row_rel_err(V, V_ref) <= TOL
    for x, y in zip(hist, hist_ref):
        assert abs(x - y) <= TOL * y


@pytest.mark.parametrize("k,p", [(64, 512), (16, 1024), (128, 256)])
def test_handover_stress(k, p):
    """Few ratings per block, many strata: three epochs in the persistent
    schedule repeat bit for bit and equal the LDS-staged sweep."""
    w = make("hs", n=4 * p + 37, m=2 * p + 11, nnz=40 * p, k=k, p=p, alpha=0.02, beta=0.05,
             epochs=3, seed=p + k + 1, structure="uniform", values="int5", rank=4)
    a = gpu_run(w, 3, v_staging=GLOBAL, schedule=2)
    b = gpu_run(w, 3, v_staging=GLOBAL, schedule=2)
    c = gpu_run(w, 3, v_staging=LDS, single=0)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert np.array_equal(a[0], c[0]) and np.array_equal(a[1], c[1])


def test_out_of_core_global_v():
    """Streaming from host memory with V in global memory equals in-core."""
    import oracle
    w = CASES["large_shape"]()
    bp, _ = oracle.bucket(w.n, w.m, w.p, w.rows, w.cols)
    budget = 3 * (int(np.diff(bp[:: w.p]).max()) + 256) * 8
    a = gpu_run(w, 2, v_staging=GLOBAL, budget=budget)
    b = gpu_run(w, 2, v_staging=LDS, single=0)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    # the streamed RMSE pass adds its fp64 partial sums in another grouping
    for x, y in zip(a[2], b[2]):
        assert abs(x - y) <= 1e-12 * y
