"""Column slices handed between the waves of a workgroup through LDS
(BGMF_OPT_LDS_HANDOVER) instead of global memory: the arithmetic of every
step is unchanged, so the factors and RMSE must be bit-identical to the
global hand-over, and match the oracle's epoch (Algorithm 1).  The cases
cover a partial last workgroup (p not a multiple of the waves per
workgroup), the wrap from row-block p - 1 to 0, empty blocks, duplicates,
several passes per block, unequal blocks and streamed strata (each chunk is
a launch of its own, so slices cross launch boundaries)."""
import numpy as np
import pytest

from helpers import oracle_run, row_rel_err
from workloads import make, make_config

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _uniform(n, m, nnz, k, p, seed, dup=False):
    if dup:  # repeated (i, j) pairs allowed
        from workloads.synth import Workload, init_factors
        rng = np.random.default_rng(seed)
        rows = rng.integers(0, n, nnz).astype(np.int32)
        cols = rng.integers(0, m, nnz).astype(np.int32)
        vals = rng.integers(1, 6, nnz).astype(np.float32)
        U0, V0 = init_factors(n, m, k, seed + 100)
        return Workload("dup", n, m, k, p, 0.01, 0.05, 1, rows, cols, vals, U0, V0)
    return make("u", n=n, m=m, nnz=nnz, k=k, p=p, alpha=0.01, beta=0.05, epochs=1, seed=seed,
                structure="uniform", values="int5", rank=4)


CASES = {
    "tiny": lambda: make_config("tiny"),
    "large_shape": lambda: make_config("large", n=48_000, m=1_800, nnz=1_000_000, p=128),
    "p_ragged_13": lambda: _uniform(1_003, 997, 40_000, 32, 13, 41),
    "p_ragged_130": lambda: _uniform(5_000, 3_000, 60_000, 64, 130, 42),
    "many_empty_blocks": lambda: _uniform(5_000, 3_000, 2_000, 16, 512, 43),
    "duplicates": lambda: _uniform(200, 150, 20_000, 16, 7, 44, dup=True),
    "k128": lambda: _uniform(2_000, 900, 50_000, 128, 32, 45),
}


def _run(w, handover, epochs=2, schedule=0, passes=1, budget=0, cuts=None):
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        if cuts is not None:
            mdl.set_cuts(*cuts)
        mdl.set_option(bgmf.BGMF_OPT_LDS_HANDOVER, handover)
        assert mdl.get_option(bgmf.BGMF_OPT_LDS_HANDOVER) == handover
        mdl.set_option(bgmf.BGMF_OPT_SCHEDULE, schedule)
        mdl.set_option(bgmf.BGMF_OPT_BLOCK_PASSES, passes)
        mdl.set_option(bgmf.BGMF_OPT_RATINGS_BUDGET, budget)
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        hist = []
        for _ in range(epochs):
            mdl.epoch(w.alpha, w.beta)
            hist.append(mdl.rmse())
        U, V = mdl.get_factors()
    return U, V, hist


def _same(a, b):
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert a[2] == b[2]


@pytest.mark.parametrize("case", sorted(CASES))
def test_bit_identical_and_oracle(case):
    w = CASES[case]()
    on = _run(w, 1)
    off = _run(w, 0)
    _same(on, off)
    U, V, hist, _, _ = oracle_run(w, 2)
    assert row_rel_err(on[0], U) <= TOL and row_rel_err(on[1], V) <= TOL
    for a, b in zip(on[2], hist):
        assert abs(a - b) <= TOL * b


@pytest.mark.parametrize("schedule", [1, 2])
def test_other_schedules(schedule):
    w = CASES["p_ragged_130"]()
    _same(_run(w, 1, schedule=schedule), _run(w, 0))


def test_passes():
    w = CASES["large_shape"]()
    _same(_run(w, 1, epochs=1, passes=3), _run(w, 0, epochs=1, passes=3))


def test_streamed():
    w = CASES["large_shape"]()
    budget = w.nnz * 8 // 5
    _same(_run(w, 1, budget=budget), _run(w, 0))


def test_unequal_blocks():
    from paper_2304_13724_amd import bgmf
    w = CASES["large_shape"]()
    cuts = bgmf.bgmf_balanced_cuts(w.n, w.m, w.p, w.rows, w.cols, 65536, 64)
    _same(_run(w, 1, cuts=cuts), _run(w, 0, cuts=cuts))


def test_handover_stress():
    """Few ratings per block, many strata: nearly every step of the epoch is
    a hand-over, three epochs."""
    p, k = 1024, 64
    w = make("hs", n=4 * p + 37, m=2 * p + 11, nnz=40 * p, k=k, p=p, alpha=0.02, beta=0.05,
             epochs=3, seed=p + k + 1, structure="uniform", values="int5", rank=4)
    on = _run(w, 1, epochs=3)
    _same(on, _run(w, 0, epochs=3))
    U, V, hist, _, _ = oracle_run(w, 3)
    assert row_rel_err(on[0], U) <= TOL and row_rel_err(on[1], V) <= TOL
