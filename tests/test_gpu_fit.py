"""Algorithm 1's outer loop (bgmf_fit: epochs until the RMSE changes by less
than delta) and the RMSE over caller-given ratings (bgmf_rmse_coo, for a
held-out split as in Table 2's test RMSE), against the oracle."""
import numpy as np
import pytest

import oracle
from helpers import row_rel_err
from workloads import make_config

pytestmark = pytest.mark.gpu

TOL = 1e-4


def _split(w, frac, seed):
    """Seeded train/test split of a workload's ratings."""
    test = np.random.default_rng(seed).random(w.nnz) < frac
    tr = (w.rows[~test], w.cols[~test], w.vals[~test])
    te = (w.rows[test], w.cols[test], w.vals[test])
    return tr, te


def _oracle_fit(w, rows, cols, vals, max_epochs, delta):
    bp, perm = oracle.bucket(w.n, w.m, w.p, rows, cols)
    U, V = w.U0.copy(), w.V0.copy()
    hist = [oracle.rmse(rows, cols, vals, U, V)]
    for _ in range(max_epochs):
        oracle.epoch(w.p, rows, cols, vals, bp, perm, U, V, w.alpha, w.beta)
        hist.append(oracle.rmse(rows, cols, vals, U, V))
        if abs(hist[-2] - hist[-1]) < delta:
            break
    return U, V, hist


@pytest.mark.parametrize("streamed", [False, True])
def test_fit_matches_oracle_loop(streamed):
    """The outer loop against the oracle's; streamed: the same run with the
    ratings streamed from host memory under a budget of two strata plus a
    margin (the epochs and RMSE passes stream every time)."""
    w = make_config("tiny")
    delta = 0.02
    U_ref, V_ref, hist_ref = _oracle_fit(w, w.rows, w.cols, w.vals, 30, delta)
    d = np.abs(np.diff(hist_ref))
    # the stopping epoch must not be decided by rounding: every change is
    # clearly above delta except the last, which is clearly below
    assert (d[:-1] > delta * 1.005).all() and d[-1] < delta * 0.995, d
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        if streamed:
            bp, _ = oracle.bucket(w.n, w.m, w.p, w.rows, w.cols)
            widest = int(np.diff(bp[:: w.p]).max())
            mdl.set_option(bgmf.BGMF_OPT_RATINGS_BUDGET, 2 * (widest + 256) * 8 + 4096)
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        assert (mdl.get_option(bgmf.BGMF_OPT_STREAM_SLOTS) > 0) == streamed
        ran, hist = mdl.fit(w.alpha, w.beta, 30, delta)
        U, V = mdl.get_factors()
    assert ran == len(hist_ref) - 1
    assert np.allclose(hist, hist_ref, rtol=TOL, atol=0)
    du, dv = row_rel_err(U, U_ref), row_rel_err(V, V_ref)
    print(f"fit, {ran} epochs: row rel err U {du:.3e} V {dv:.3e}", flush=True)
    assert du <= TOL and dv <= TOL


def test_heldout_rmse():
    w = make_config("tiny")
    (r, c, x), (rt, ct, xt) = _split(w, 0.1, 5)
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(r, c, x)
        for _ in range(3):
            mdl.epoch(w.alpha, w.beta)
        train = mdl.rmse()
        train_coo = mdl.rmse_coo(r, c, x)
        test = mdl.rmse_coo(rt, ct, xt)
        U, V = mdl.get_factors()
    # the same factors: only the order of the fp32 dots differs
    assert abs(train_coo - train) <= 1e-6 * train
    assert abs(test - oracle.rmse(rt, ct, xt, U, V)) <= 1e-6 * test
    # against factors trained by the oracle on the same split
    bp, perm = oracle.bucket(w.n, w.m, w.p, r, c)
    Uo, Vo = w.U0.copy(), w.V0.copy()
    for _ in range(3):
        oracle.epoch(w.p, r, c, x, bp, perm, Uo, Vo, w.alpha, w.beta)
    ref = oracle.rmse(rt, ct, xt, Uo, Vo)
    assert abs(test - ref) <= TOL * ref
    assert test > train  # held-out ratings fit worse than the training ones


def test_fit_reports_divergence():
    w = make_config("tiny")
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.fit(5.0, 0.0, 10, 1e-6)
        assert ei.value.code == bgmf.BGMF_E_NONFINITE
        assert 1 <= ei.value.epochs_run <= 10
        assert np.isfinite(ei.value.rmse_history[0])
        assert not np.isfinite(ei.value.rmse_history[-1])


def test_fit_and_rmse_coo_argument_errors():
    w = make_config("tiny")
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.rmse_coo(w.rows, w.cols, w.vals)
        assert ei.value.code == bgmf.BGMF_E_STATE
        mdl.set_factors(w.U0, w.V0)
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.fit(w.alpha, w.beta, 5, 0.01)  # no ratings loaded
        assert ei.value.code == bgmf.BGMF_E_STATE
        mdl.load_coo(w.rows, w.cols, w.vals)
        for me, d in [(0, 0.1), (5, -1.0), (5, float("nan"))]:
            with pytest.raises(bgmf.BgmfError) as ei:
                mdl.fit(w.alpha, w.beta, me, d)
            assert ei.value.code == bgmf.BGMF_E_ARG
        bad = w.cols.copy()
        bad[3] = w.m
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.rmse_coo(w.rows, bad, w.vals)
        assert ei.value.code == bgmf.BGMF_E_RANGE
        badv = w.vals.copy()
        badv[0] = np.inf
        with pytest.raises(bgmf.BgmfError) as ei:
            mdl.rmse_coo(w.rows, w.cols, badv)
        assert ei.value.code == bgmf.BGMF_E_NONFINITE
