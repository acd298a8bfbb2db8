"""The allocation-free entry point bgmf_rmse_coo_dev against bgmf_rmse_coo:
the same RMSE over ratings given in device memory (PyTorch tensors), with
no allocation by the library, on two calls in a row (the second with a
smaller input), and its device-side argument checks."""
import numpy as np
import pytest

import oracle
from workloads import make_config

pytestmark = pytest.mark.gpu


def _dev(mdl, rows_t, cols_t, vals_t):
    from paper_2304_13724_amd import bgmf
    return bgmf.bgmf_rmse_coo_dev(mdl.h, rows_t.data_ptr(), cols_t.data_ptr(), vals_t.data_ptr(),
                                  rows_t.shape[0])


def test_rmse_coo_dev_matches_rmse_coo_without_allocating():
    import torch
    from paper_2304_13724_amd import bgmf
    torch.cuda.set_device(0)
    w = make_config("tiny")
    rng = np.random.default_rng(7)
    U = (w.U0 + rng.normal(0, 0.05, w.U0.shape)).astype(np.float32)
    V = (w.V0 + rng.normal(0, 0.05, w.V0.shape)).astype(np.float32)
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_factors(U, V)
        before = mdl.get_option(bgmf.BGMF_OPT_ALLOC_COUNT)
        for sl in (slice(0, w.nnz), slice(1000, 31000)):  # the second call is smaller
            rows, cols, vals = w.rows[sl], w.cols[sl], w.vals[sl]
            rows_t = torch.from_numpy(np.ascontiguousarray(rows)).to("cuda:0")
            cols_t = torch.from_numpy(np.ascontiguousarray(cols)).to("cuda:0")
            vals_t = torch.from_numpy(np.ascontiguousarray(vals)).to("cuda:0")
            torch.cuda.synchronize()
            a0 = mdl.get_option(bgmf.BGMF_OPT_ALLOC_COUNT)
            r_dev = _dev(mdl, rows_t, cols_t, vals_t)
            assert mdl.get_option(bgmf.BGMF_OPT_ALLOC_COUNT) == a0  # nothing allocated
            r_host = mdl.rmse_coo(rows, cols, vals)
            r_ref = oracle.rmse(rows, cols, vals, U, V)
            print(f"n={rows.shape[0]}: dev {r_dev!r} host {r_host!r} oracle {r_ref!r}", flush=True)
            assert r_dev == r_host  # same kernel, same fixed reduction order
            assert abs(r_dev - r_ref) <= 1e-6 * r_ref
        assert mdl.get_option(bgmf.BGMF_OPT_ALLOC_COUNT) > before  # only bgmf_rmse_coo's


def test_rmse_coo_dev_device_checks():
    """An index outside the matrix or a non-finite value, in device memory,
    is reported (the kernel skips such ratings without reading factors),
    and the next call starts from a cleared error word."""
    import torch
    from paper_2304_13724_amd import bgmf
    torch.cuda.set_device(0)
    w = make_config("tiny")
    rows = np.ascontiguousarray(w.rows[:5000])
    cols = np.ascontiguousarray(w.cols[:5000])
    vals = np.ascontiguousarray(w.vals[:5000])
    with bgmf.Model(w.n, w.m, w.k, w.p) as mdl:
        mdl.set_factors(w.U0, w.V0)
        good = [torch.from_numpy(a).to("cuda:0") for a in (rows, cols, vals)]
        bad_row = good[0].clone()
        bad_row[17] = w.n
        bad_val = good[2].clone()
        bad_val[4000] = float("nan")
        torch.cuda.synchronize()
        with pytest.raises(bgmf.BgmfError) as ei:
            _dev(mdl, bad_row, good[1], good[2])
        assert ei.value.code == bgmf.BGMF_E_RANGE
        with pytest.raises(bgmf.BgmfError) as ei:
            _dev(mdl, good[0], good[1], bad_val)
        assert ei.value.code == bgmf.BGMF_E_NONFINITE
        assert _dev(mdl, *good) == mdl.rmse_coo(rows, cols, vals)
        with pytest.raises(bgmf.BgmfError) as ei:
            bgmf.bgmf_rmse_coo_dev(mdl.h, good[0].data_ptr(), good[1].data_ptr(),
                                   good[2].data_ptr(), 1 << 31)
        assert ei.value.code == bgmf.BGMF_E_ARG
