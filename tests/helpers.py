"""Shared helpers for the GPU parity tests (comparison metrics, runners)."""
import numpy as np

import oracle


def row_rel_err(a: np.ndarray, b: np.ndarray) -> float:
    """max over rows of |a_i - b_i|_inf / |b_i|_inf (rows of b that are all
    zero use an absolute error)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    num = np.abs(a - b).max(axis=1)
    den = np.abs(b).max(axis=1)
    den = np.where(den > 0, den, 1.0)
    return float((num / den).max()) if a.size else 0.0


def oracle_run(w, epochs, threads=1, layout=None):
    """Bucket with the oracle and run ``epochs`` epochs; returns
    (U, V, rmse_history, block_ptr, perm)."""
    if layout is None:
        bp, perm = oracle.bucket(w.n, w.m, w.p, w.rows, w.cols)
    else:
        bp, perm = layout
    U, V = w.U0.copy(), w.V0.copy()
    hist = []
    for _ in range(epochs):
        oracle.epoch_mt(w.p, w.rows, w.cols, w.vals, bp, perm, U, V, w.alpha, w.beta, threads)
        hist.append(oracle.rmse(w.rows, w.cols, w.vals, U, V))
    return U, V, hist, bp, perm


def gpu_run(w, epochs, schedule=0, xcd_remap=1, v_staging=0, budget=0, single=1):
    """Run the HIP path through the C ABI; returns (U, V, rmse_history, block_ptr, perm).
    ``v_staging``: 0 automatic, 1 V slice in LDS, 2 V in global memory;
    ``budget``: ratings budget in bytes (0 = all ratings on the device);
    ``single``: BGMF_OPT_SINGLE_COLUMN (0 when a run with V in LDS is compared
    bit for bit with one with V in global memory, which has no folded step)."""
    from paper_2304_13724_amd import bgmf
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_option(bgmf.BGMF_OPT_SCHEDULE, schedule)
        mdl.set_option(bgmf.BGMF_OPT_XCD_REMAP, xcd_remap)
        mdl.set_option(bgmf.BGMF_OPT_V_STAGING, v_staging)
        mdl.set_option(bgmf.BGMF_OPT_RATINGS_BUDGET, budget)
        mdl.set_option(bgmf.BGMF_OPT_SINGLE_COLUMN, single)
        mdl.set_factors(w.U0, w.V0)
        mdl.load_coo(w.rows, w.cols, w.vals)
        bp, perm = mdl.get_layout()
        hist = []
        for _ in range(epochs):
            mdl.epoch(w.alpha, w.beta)
            hist.append(mdl.rmse())
        U, V = mdl.get_factors()
    return U, V, hist, bp, perm
