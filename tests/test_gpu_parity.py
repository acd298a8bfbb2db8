"""GPU parity: the HIP path through the C ABI against the CPU oracle.

Bar: bucketing (block_ptr, perm) bit-exact; U and V within 1e-4 row-wise
relative error after one epoch; RMSE within 1e-4 relative after every
epoch.  The GPU sums dot products in a different order and with fused
multiply-adds, so floating-point results are compared by tolerance.
"""
import numpy as np
import pytest

import oracle
from helpers import gpu_run, oracle_run, row_rel_err
from workloads import make, make_config

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _uniform(n, m, nnz, k, p, seed, alpha=0.01, beta=0.05, dup=False):
    if dup:
        rng = np.random.default_rng(seed)
        rows = rng.integers(0, n, nnz).astype(np.int32)
        cols = rng.integers(0, m, nnz).astype(np.int32)
        vals = rng.integers(1, 6, nnz).astype(np.float32)
        from workloads.synth import Workload, init_factors
        U0, V0 = init_factors(n, m, k, seed + 100)
        return Workload("dup", n, m, k, p, alpha, beta, 1, rows, cols, vals, U0, V0)
    return make("u", n=n, m=m, nnz=nnz, k=k, p=p, alpha=alpha, beta=beta, epochs=1, seed=seed,
                structure="uniform", values="int5", rank=4)


CASES = {
    "tiny": lambda: make_config("tiny"),
    "medium_shape": lambda: make_config("medium", n=7_000, m=1_000, nnz=300_000, p=32),
    "large_shape": lambda: make_config("large", n=48_000, m=1_800, nnz=1_000_000, p=128),
    "p1": lambda: _uniform(300, 200, 5_000, 16, 1, 7),
    "p_eq_n": lambda: _uniform(96, 96, 3_000, 32, 96, 8),
    "many_empty_blocks": lambda: _uniform(5_000, 3_000, 2_000, 16, 512, 9),
    "duplicates": lambda: _uniform(200, 150, 20_000, 16, 7, 10, dup=True),
    "single_rating": lambda: _uniform(10, 10, 1, 16, 3, 11),
    "ragged_p": lambda: _uniform(1_003, 997, 40_000, 32, 13, 12),
    # the widest blocks a record can index: 65,536 rows by 65,536 columns
    "widest_blocks": lambda: _uniform(131_072, 131_072, 300_000, 16, 2, 13),
    # degenerate shapes: a 1 x 1 matrix, one user, one item
    "one_cell": lambda: _uniform(1, 1, 1, 16, 1, 15),
    "one_row": lambda: _uniform(1, 500, 400, 32, 1, 16),
    "one_column": lambda: _uniform(500, 1, 400, 32, 1, 17),
}


@pytest.mark.parametrize("case", sorted(CASES))
def test_bucketing_bit_exact(case):
    w = CASES[case]()
    bp_ref, perm_ref = oracle.bucket(w.n, w.m, w.p, w.rows, w.cols)
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.load_coo(w.rows, w.cols, w.vals)
        bp, perm = mdl.get_layout()
    assert np.array_equal(bp, bp_ref)
    assert np.array_equal(perm, perm_ref)


@pytest.mark.parametrize("case", sorted(CASES))
@pytest.mark.parametrize("schedule", [0, 1])
def test_one_epoch_parity(case, schedule):
    w = CASES[case]()
    U_ref, V_ref, hist_ref, _, _ = oracle_run(w, 1)
    U, V, hist, _, _ = gpu_run(w, 1, schedule=schedule)
    assert row_rel_err(U, U_ref) <= TOL
    assert row_rel_err(V, V_ref) <= TOL
    assert abs(hist[0] - hist_ref[0]) <= TOL * hist_ref[0]


def test_largest_grid():
    """p = 8192, the largest grid: 67M block slots, 8192 strata, mostly
    empty blocks; bucketing bit-exact and one epoch against the oracle."""
    w = _uniform(16_384, 16_384, 200_000, 16, 8192, 14)
    bp_ref, perm_ref = oracle.bucket(w.n, w.m, w.p, w.rows, w.cols)
    U_ref, V_ref, hist_ref, _, _ = oracle_run(w, 1, layout=(bp_ref, perm_ref))
    U, V, hist, bp, perm = gpu_run(w, 1)
    assert np.array_equal(bp, bp_ref) and np.array_equal(perm, perm_ref)
    assert row_rel_err(U, U_ref) <= TOL and row_rel_err(V, V_ref) <= TOL
    assert abs(hist[0] - hist_ref[0]) <= TOL * hist_ref[0]


@pytest.mark.parametrize("k", [16, 32, 48, 64, 80, 128, 256])
def test_factor_widths(k):
    w = make_config("medium", n=3_000, m=700, nnz=60_000, p=16, k=k)
    U_ref, V_ref, hist_ref, _, _ = oracle_run(w, 2)
    U, V, hist, _, _ = gpu_run(w, 2)
    assert row_rel_err(U, U_ref) <= TOL
    assert row_rel_err(V, V_ref) <= TOL
    for a, b in zip(hist, hist_ref):
        assert abs(a - b) <= TOL * b


def test_tiny_config_all_epochs():
    """Tiny planted low-rank workload, its full 5 epochs: RMSE after every
    epoch and final factors against the oracle."""
    w = make_config("tiny")
    U_ref, V_ref, hist_ref, _, _ = oracle_run(w, w.epochs)
    U, V, hist, _, _ = gpu_run(w, w.epochs)
    for a, b in zip(hist, hist_ref):
        assert abs(a - b) <= TOL * b, (hist, hist_ref)
    assert all(y < x for x, y in zip(hist, hist[1:]))
    du, dv = row_rel_err(U, U_ref), row_rel_err(V, V_ref)
    print(f"tiny, 5 epochs: row rel err U {du:.3e} V {dv:.3e}", flush=True)
    assert du <= TOL and dv <= TOL


def test_xcd_remap_off_matches():
    w = CASES["large_shape"]()
    a = gpu_run(w, 1, xcd_remap=1)
    b = gpu_run(w, 1, xcd_remap=0)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_run_to_run_bit_identical():
    w = CASES["medium_shape"]()
    a = gpu_run(w, 2)
    b = gpu_run(w, 2)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert a[2] == b[2]
    c = gpu_run(w, 2, schedule=1)
    assert np.array_equal(a[0], c[0]) and np.array_equal(a[1], c[1])


def test_resume_is_bit_identical():
    """get_factors after epoch 1, a fresh handle with those factors for
    epoch 2 == two epochs on one handle (an epoch carries no hidden state)."""
    from paper_2304_13724_amd import bgmf
    w = CASES["medium_shape"]()
    U2, V2, _, _, _ = gpu_run(w, 2)
    with bgmf.Model(w.n, w.m, w.k, w.p) as a:
        a.set_factors(w.U0, w.V0)
        a.load_coo(w.rows, w.cols, w.vals)
        a.epoch(w.alpha, w.beta)
        U1, V1 = a.get_factors()
    with bgmf.Model(w.n, w.m, w.k, w.p) as b:
        b.set_factors(U1, V1)
        b.load_coo(w.rows, w.cols, w.vals)
        b.epoch(w.alpha, w.beta)
        Ur, Vr = b.get_factors()
    assert np.array_equal(Ur, U2) and np.array_equal(Vr, V2)


def test_errors_and_states():
    from paper_2304_13724_amd import bgmf
    w = make_config("tiny")
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.epoch(0.01, 0.05)
        assert ei.value.code == bgmf.BGMF_E_STATE
        mdl.set_factors(w.U0, w.V0)
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.rmse()
        assert ei.value.code == bgmf.BGMF_E_STATE
        bad = w.rows.copy()
        bad[5] = w.n
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.load_coo(bad, w.cols, w.vals)
        assert ei.value.code == bgmf.BGMF_E_RANGE
        badv = w.vals.copy()
        badv[3] = np.nan
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.load_coo(w.rows, w.cols, badv)
        assert ei.value.code == bgmf.BGMF_E_NONFINITE
        mdl.load_coo(w.rows, w.cols, w.vals)
        for a, b in [(0.0, 0.05), (-1.0, 0.0), (0.01, -0.1), (float("nan"), 0.0)]:
            with pytest.raises(bgmf.BgmfError) as ei:
                mdl.epoch(a, b)
            assert ei.value.code == bgmf.BGMF_E_ARG
        mdl.epoch(w.alpha, w.beta)
        r = mdl.rmse()
        assert np.isfinite(r)


def test_wait_limit_error_path():
    """A zero wait limit on a schedule that is sure to wait: with p = 2,
    row-block 1's block of stratum 0 holds 200,000 ratings and row-block 0's
    none, so in stratum 1 wave 0 needs the column-block that wave 1 is still
    sweeping (some 10 ms), and its first poll finds it unfinished.  The wait
    gives up, the kernel still exits, the error is reported as
    BGMF_E_TIMEOUT, and the handle keeps working afterwards."""
    from paper_2304_13724_amd import bgmf
    from workloads.synth import Workload, init_factors
    rng = np.random.default_rng(11)
    n = m = 128
    heavy = 200_000
    rows = np.r_[rng.integers(64, 128, heavy), rng.integers(0, 64, 100)].astype(np.int32)
    cols = np.r_[rng.integers(64, 128, heavy), rng.integers(64, 128, 100)].astype(np.int32)
    vals = rng.integers(1, 6, heavy + 100).astype(np.float32)
    U0, V0 = init_factors(n, m, 16, 5)
    w = Workload("wait", n, m, 16, 2, 0.002, 0.05, 1, rows, cols, vals, U0, V0)
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        assert mdl.get_option(bgmf.BGMF_OPT_PLACEMENT) & 4  # one persistent launch
        mdl.set_option(bgmf.BGMF_OPT_WAIT_LIMIT_US, 0)
        mdl.epoch(w.alpha, w.beta)
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.sync()
        assert ei.value.code == bgmf.BGMF_E_TIMEOUT
        mdl.set_option(bgmf.BGMF_OPT_WAIT_LIMIT_US, 10_000_000)
        mdl.set_factors(w.U0, w.V0)
        mdl.epoch(w.alpha, w.beta)
        mdl.sync()
        U, V = mdl.get_factors()
    U_ref, V_ref, _, _, _ = oracle_run(w, 1)
    assert row_rel_err(U, U_ref) <= TOL and row_rel_err(V, V_ref) <= TOL


@pytest.mark.parametrize("k,p", [(64, 512), (16, 1024), (128, 256)])
def test_handover_stress(k, p):
    """Many strata with few ratings per block: every epoch is mostly
    column-slice hand-overs between neighbouring waves.  Three epochs must
    match the oracle and repeat bit for bit."""
    w = make("hs", n=4 * p + 37, m=2 * p + 11, nnz=40 * p, k=k, p=p, alpha=0.02, beta=0.05,
             epochs=3, seed=p + k, structure="uniform", values="int5", rank=4)
    U_ref, V_ref, hist_ref, _, _ = oracle_run(w, 3)
    a = gpu_run(w, 3)
    b = gpu_run(w, 3)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])
    assert row_rel_err(a[0], U_ref) <= TOL and row_rel_err(a[1], V_ref) <= TOL
    for x, y in zip(a[2], hist_ref):
        assert abs(x - y) <= TOL * y
